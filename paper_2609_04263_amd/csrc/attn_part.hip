// Decode attention split kernels of one instance family, selected at build
// time: KVQ_PART_D (head size 64, 128 or 256), KVQ_PART_M16 (fp16 scales
// and offsets) and KVQ_PART_PC (per-channel keys).  The build compiles this
// file once per family, so the families compile in parallel.
#include "attn_impl.h"

#if !defined(KVQ_PART_D) || !defined(KVQ_PART_M16) || !defined(KVQ_PART_PC)
#error "attn_part.hip is compiled once per family with KVQ_PART_D, KVQ_PART_M16 and KVQ_PART_PC defined"
#endif

#define KVQ_CAT2(a, b, c, d) a##_##b##_##c##_##d
#define KVQ_CAT(a, b, c, d) KVQ_CAT2(a, b, c, d)

namespace kvq {

hipError_t KVQ_CAT(launch_split, KVQ_PART_D, KVQ_PART_M16, KVQ_PART_PC)(const AttnParams& p, hipStream_t stream)
{
    return attn::launch_split_family<KVQ_PART_D, KVQ_PART_M16 != 0, KVQ_PART_PC != 0>(p, stream);
}

int KVQ_CAT(resident_split, KVQ_PART_D, KVQ_PART_M16, KVQ_PART_PC)(const AttnParams& p)
{
    return attn::resident_family<KVQ_PART_D, KVQ_PART_M16 != 0, KVQ_PART_PC != 0>(p);
}

}  // namespace kvq
