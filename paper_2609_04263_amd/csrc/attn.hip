// Decode attention: split planning and dispatch by head dimension.  The
// kernels live in attn_impl.h and are instantiated in one translation unit
// per head dimension (attn_d64.hip, attn_d128.hip, attn_d256.hip).

#include "attn_impl.h"

namespace kvq {

hipError_t launch_decode_64(const AttnParams& p, hipStream_t stream);
hipError_t launch_decode_128(const AttnParams& p, hipStream_t stream);
hipError_t launch_decode_256(const AttnParams& p, hipStream_t stream);

// Split planning.  Each wave streams every fourth block of its split with
// the next block's loads in flight, so a split may be long; splits only
// exist to give the 256 compute units about kTargetGroups workgroups (a few
// resident per CU, so that one's loads overlap another's arithmetic).
// Blocks per split are a multiple of the wave count.
constexpr int kTargetGroups = 1024;

static int splits_wanted(int B, int H)
{
    const int units = B * H;
    const int s = (kTargetGroups + units - 1) / units;
    return s < 1 ? 1 : s;
}

void decode_plan(int B, int H, int D, const kvq_format& f, int nq, int* S_q, int* bps)
{
    (void)D;
    (void)f;
    const int nblk = (nq + 31) / 32;
    const int sb = attn::kWaves;
    if (nblk == 0) {
        *S_q = 0;
        *bps = sb;
        return;
    }
    int per = (nblk + splits_wanted(B, H) - 1) / splits_wanted(B, H);
    per = (per + sb - 1) / sb * sb;
    *bps = per;
    *S_q = (nblk + per - 1) / per;
}

int decode_split_bound(int B, int H, int D, const kvq_format& f, int nq)
{
    // S_q = ceil(nblk / per) with per >= nblk / splits_wanted.
    (void)D;
    (void)f;
    (void)nq;
    return splits_wanted(B, H);
}

size_t decode_lds_bytes(int D, const kvq_format& f, int G)
{
    // Per-wave metadata buffers; the query rows and the final merge reuse
    // the same memory.
    const int nvg = D / f.v_group;
    size_t need = (size_t)attn::kWaves * 1024 * attn::meta_loads(D, f.k_axis == KVQ_PER_CHANNEL, nvg);
    const size_t q = 16 * (size_t)D * sizeof(float);
    const size_t merge = (2 * attn::kWaves * 16 + (size_t)attn::kWaves * G * D) * sizeof(float);
    if (q > need)
        need = q;
    if (merge > need)
        need = merge;
    return need;
}

hipError_t launch_decode(const AttnParams& p, int D, hipStream_t stream)
{
    switch (D) {
    case 64:
        return launch_decode_64(p, stream);
    case 128:
        return launch_decode_128(p, stream);
    case 256:
        return launch_decode_256(p, stream);
    default:
        return hipErrorInvalidValue;
    }
}

}  // namespace kvq
