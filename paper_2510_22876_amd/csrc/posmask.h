// Position ids and attention mask of invariant I2 (EqSpec, arXiv 2510.22876,
// Section 3.1) for one left-padded row: column j is content when j >= pad,
// and a content column's position id is its index within the row's content.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace specdec {

// Writes columns [cb*4*kTpb, (cb+1)*4*kTpb) of the row, clipped to `width`:
// mask = (j >= pad), pos = max(0, j - pad).  `pad` and `width` are validated
// by the caller.
template <int kTpb>
__device__ __forceinline__ void posmask_cols(uint32_t cb, int64_t* prow, uint8_t* mrow, int64_t pad, int64_t width) {
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int64_t j = static_cast<int64_t>(cb) * (4 * kTpb) + q * kTpb + threadIdx.x;
    if (j < width) {
      const bool content = j >= pad;
      prow[j] = content ? j - pad : 0;
      mrow[j] = content ? 1 : 0;
    }
  }
}

}  // namespace specdec
