// Decode attention kernels for head_dim 64.
#include "attn_impl.h"

namespace kvq {

hipError_t launch_decode_64(const AttnParams& p, hipStream_t stream)
{
    return attn::launch_decode_d<64>(p, stream);
}

int decode_resident_64(const AttnParams& p)
{
    return attn::resident_d<64>(p);
}

}  // namespace kvq
