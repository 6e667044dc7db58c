// The decode partials kernel for 4 query heads per KV head, compiled apart from kvc_decode.hip
// (which defines it and declares this instantiation external) so that the largest instantiations
// of the kernel build in parallel. CDNA4 / gfx950 only.
#define KVC_DECODE_PARTIALS_UNIT
#include "kvc_decode.hip"

namespace kvc {
template __global__ void decode_partial_kernel<4>(DevSide, DevSide, const v4i*, const float4*, const int32_t*, int, int,
                                                  int, int, int, float*);
}  // namespace kvc
