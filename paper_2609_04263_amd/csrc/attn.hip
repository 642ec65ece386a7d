// Decode attention: split planning and dispatch by head dimension.  The
// kernels live in attn_impl.h and are instantiated in one translation unit
// per head dimension (attn_d64.hip, attn_d128.hip, attn_d256.hip).

#include "attn_impl.h"

namespace kvq {

hipError_t launch_decode_64(const AttnParams& p, hipStream_t stream);
hipError_t launch_decode_128(const AttnParams& p, hipStream_t stream);
hipError_t launch_decode_256(const AttnParams& p, hipStream_t stream);
int decode_resident_64(const AttnParams& p);
int decode_resident_128(const AttnParams& p);
int decode_resident_256(const AttnParams& p);

// Split planning.  Each wave streams every fourth block of its split with
// the next block's loads in flight, so a split may be long; splits exist to
// fill the chip with one round of resident workgroups (a second, partial
// round would run at a fraction of the occupancy).  Blocks per split are a
// multiple of the wave count.  The target never exceeds kMaxGroups, which
// bounds the workspace.
constexpr int kMaxGroups = 1024;

static int splits_for(int B, int H, int groups)
{
    const int units = B * H;
    if (groups > kMaxGroups)
        groups = kMaxGroups;
    const int s = groups / units;
    return s < 1 ? 1 : s;
}

static int compute_units()
{
    // cached per device (device ids below 64; others are queried each time)
    static std::atomic<int> cached[64];
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess)
        return 256;
    if (dev >= 0 && dev < 64 && (cus = cached[dev].load(std::memory_order_relaxed)) > 0)
        return cus;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus < 1)
        cus = 256;
    if (dev >= 0 && dev < 64)
        cached[dev].store(cus, std::memory_order_relaxed);
    return cus;
}

int decode_target_groups(const AttnParams& p, int D)
{
    const int cus = compute_units();
    int per = 1;
    switch (D) {
    case 64:
        per = decode_resident_64(p);
        break;
    case 128:
        per = decode_resident_128(p);
        break;
    case 256:
        per = decode_resident_256(p);
        break;
    default:
        break;
    }
    return per * cus;
}

void decode_plan(int B, int H, int groups, int nq, int* S_q, int* bps)
{
    const int nblk = (nq + 31) / 32;
    const int sb = attn::kWaves;
    if (nblk == 0) {
        *S_q = 0;
        *bps = sb;
        return;
    }
    const int s = splits_for(B, H, groups);
    int per = (nblk + s - 1) / s;
    per = (per + sb - 1) / sb * sb;
    *bps = per;
    *S_q = (nblk + per - 1) / per;
}

int decode_split_bound(int B, int H)
{
    // S_q = ceil(nblk / per) with per >= nblk / splits_for(...) and the
    // target capped at kMaxGroups.
    const int units = B * H;
    const int s = kMaxGroups / units;
    return s < 1 ? 1 : s;
}

size_t decode_lds_bytes(int D, const kvq_format& f, int G)
{
    // Per-wave metadata buffers; the query rows and the final merge reuse
    // the same memory.
    const int nvg = D / f.v_group;
    size_t need = (size_t)attn::kWaves * 2048 * attn::meta_pairs(D, nvg);
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
