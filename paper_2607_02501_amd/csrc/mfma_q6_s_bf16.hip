// mfma_q6_s_bf16.hip -- the tile kernel of the matrix-core path (mfma_tile.h)
// instantiated for Q6_S weights and bfloat16 activations (ops of more than 128 rows;
// smaller ones take mm_q6_kernel).
#include "mfma_tile.h"

namespace eb {

template hipError_t mfma_tile_launch<EB_Q6_S, EB_BF16>(int, bool, const void *, int64_t, int64_t,
                                                  const void *, int64_t, void *, int32_t,
                                                  const Fuse &, int, int, float *, int64_t,
                                                  hipStream_t);
template hipError_t mfma_tile_launch_grouped<EB_Q6_S, EB_BF16>(int, const GOp *, const int2 *, int64_t,
                                                          hipStream_t);

}  // namespace eb
