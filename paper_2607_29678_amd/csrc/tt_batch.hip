// Batches (Sec. 4.2: documents are concatenated; no piece or token crosses a
// document boundary): the output offset of every document, once the tile
// kernel has placed all tokens.
#include "tt_internal.h"

namespace tt {

// Batch: output offset of every document.  A non-empty document starts a
// unit; its processing tile recorded where the unit's tokens begin among the
// tile's outputs.  Offsets at the end of the text are the total.
__global__ void doc_offsets_kernel(Work w) {
  const int64_t T = *w.out_len;
  for (int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; j <= w.n_docs;
       j += (int64_t)gridDim.x * blockDim.x) {
    const int64_t d = w.doc_off[j];
    int64_t o = 0;
    if (T >= 0) {
      if (d >= (int64_t)w.n) {
        o = T;
      } else {
        const uint32_t ut = w.unit_tile[d];
        o = ut < w.n_tiles ? (int64_t)w.tile_pre[ut] + w.unit_pos[d] : 0;
      }
    }
    w.out_doc_off[j] = o;
  }
}

hipError_t launch_doc_offsets(const Work& w, hipStream_t s) {
  uint32_t blocks = (uint32_t)((w.n_docs + 1 + 255) / 256);
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(doc_offsets_kernel, dim3(blocks), dim3(256), 0, s, w);
  return hipGetLastError();
}

}  // namespace tt
