// Decode attention: split planning, dispatch to the split-kernel families
// (attn_part.hip, one object per head size x metadata width x key axis) and
// the merge kernels.

#include "attn_impl.h"

namespace kvq {

#define KVQ_FAMILY(D, M, P)                                                     \
    hipError_t launch_split_##D##_##M##_##P(const AttnParams& p, hipStream_t s); \
    int resident_split_##D##_##M##_##P(const AttnParams& p);
#define KVQ_FAMILIES(D) KVQ_FAMILY(D, 0, 0) KVQ_FAMILY(D, 0, 1) KVQ_FAMILY(D, 1, 0) KVQ_FAMILY(D, 1, 1)
KVQ_FAMILIES(64)
KVQ_FAMILIES(128)
KVQ_FAMILIES(256)
#undef KVQ_FAMILIES
#undef KVQ_FAMILY

namespace {

typedef hipError_t (*SplitLaunch)(const AttnParams&, hipStream_t);
typedef int (*SplitResident)(const AttnParams&);

// family index: (D slot) * 4 + meta16 * 2 + per-channel keys
const SplitLaunch kLaunch[12] = {
    launch_split_64_0_0,  launch_split_64_0_1,  launch_split_64_1_0,  launch_split_64_1_1,
    launch_split_128_0_0, launch_split_128_0_1, launch_split_128_1_0, launch_split_128_1_1,
    launch_split_256_0_0, launch_split_256_0_1, launch_split_256_1_0, launch_split_256_1_1};
const SplitResident kResident[12] = {
    resident_split_64_0_0,  resident_split_64_0_1,  resident_split_64_1_0,  resident_split_64_1_1,
    resident_split_128_0_0, resident_split_128_0_1, resident_split_128_1_0, resident_split_128_1_1,
    resident_split_256_0_0, resident_split_256_0_1, resident_split_256_1_0, resident_split_256_1_1};

int family(const AttnParams& p, int D)
{
    const int slot = D == 64 ? 0 : D == 128 ? 1 : D == 256 ? 2 : -1;
    if (slot < 0)
        return -1;
    return slot * 4 + (p.meta16 ? 2 : 0) + (p.k_axis == KVQ_PER_CHANNEL ? 1 : 0);
}

}  // namespace

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
    const int f = family(p, D);
    const int per = f < 0 ? 1 : kResident[f](p);
    return per * compute_units();
}

void decode_plan(int B, int H, int waves, int groups, int nq, int* S_q, int* bps)
{
    const int nblk = (nq + 31) / 32;
    const int sb = waves;
    if (nblk == 0) {
        // no coded tokens: one split walks the fp16 tokens
        *S_q = 1;
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

int decode_waves(int D, const kvq_format& f)
{
    return attn::waves_for(D, f.k_axis == KVQ_PER_CHANNEL, f.k_bits, f.v_bits);
}

size_t decode_lds_bytes(int D, const kvq_format& f, int G)
{
    // the layout is described in attn_impl.h
    const int nvg = D / f.v_group, np = attn::meta_pairs(D, nvg);
    const bool perch = f.k_axis == KVQ_PER_CHANNEL, fp16 = f.flush || f.sink;
    const int W = decode_waves(D, f);
    const size_t need = attn::lds_waves(D, perch, G) + (size_t)W * attn::lds_per_wave(D, np, perch, G, fp16);
    const size_t merge = (2 * (size_t)W * 16 + (size_t)W * G * D) * sizeof(float);
    return merge > need ? merge : need;
}

hipError_t launch_decode(const AttnParams& p, int D, hipStream_t stream)
{
    const int f = family(p, D);
    if (f < 0)
        return hipErrorInvalidValue;
    const hipError_t e = kLaunch[f](p, stream);
    if (e != hipSuccess || p.S_tot == 1)
        return e;
    switch (D) {
    case 64:
        return attn::launch_merge<64>(p, stream);
    case 128:
        return attn::launch_merge<128>(p, stream);
    default:
        return attn::launch_merge<256>(p, stream);
    }
}

}  // namespace kvq
