// Decode attention kernels for head_dim 256.
#include "attn_impl.h"

namespace kvq {

hipError_t launch_decode_256(const AttnParams& p, hipStream_t stream)
{
    return attn::launch_decode_d<256>(p, stream);
}

int decode_resident_256(const AttnParams& p)
{
    return attn::resident_d<256>(p);
}

}  // namespace kvq
