// Decode attention kernels for head_dim 128.
#include "attn_impl.h"

namespace kvq {

hipError_t launch_decode_128(const AttnParams& p, hipStream_t stream)
{
    return attn::launch_decode_d<128>(p, stream);
}

int decode_resident_128(const AttnParams& p)
{
    return attn::resident_d<128>(p);
}

}  // namespace kvq
