// Output placement: every tile staged its outputs (token IDs, or piece
// offsets for the split export) contiguously where its bytes begin; the emit
// kernel moves each tile's block to its place in the dense output, which is
// the exclusive prefix of the tiles' counts (the output compaction that ends
// the pipeline of Sec. 4.2), and maps internal token IDs to the caller's.
// The last tile writes the output length, or the error of the call.
#include "tt_internal.h"

namespace tt {

namespace {

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v += (uint32_t)__shfl_xor((int)v, d, 64);
  return v;
}

__device__ __forceinline__ uint32_t wave_incl_sum(uint32_t v, int lane) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const uint32_t o = (uint32_t)__shfl_up((int)v, d, 64);
    if (lane >= d) v += o;
  }
  return v;
}

}  // namespace

// One block per tile.  With `direct`, the block sums the counts of the
// earlier tiles itself (few tiles); otherwise tile_scan_kernel has written the
// prefixes to tile_pre.
template <int MODE>
__global__ __launch_bounds__(EMIT_THREADS) void emit_kernel(Work w, DevTables tb, int direct) {
  __shared__ uint32_t s_part[EMIT_THREADS / 64];
  const uint32_t t = blockIdx.x;
  const int tid = (int)threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  uint32_t prefix;
  if (direct) {
    uint32_t acc = 0;
    for (uint32_t u = (uint32_t)tid; u < t; u += EMIT_THREADS) acc += w.tile_cnt[u];
    acc = wave_sum(acc);
    if (lane == 0) s_part[wave] = acc;
    __syncthreads();
    prefix = 0;
#pragma unroll
    for (int v = 0; v < (int)(EMIT_THREADS / 64); ++v) prefix += s_part[v];
    if (w.doc_off != nullptr && tid == 0) w.tile_pre[t] = prefix;
  } else {
    prefix = w.tile_pre[t];
  }
  const uint32_t cnt = w.tile_cnt[t];
  const uint32_t* __restrict__ src = w.stage + w.tile_base[t];
  int32_t* __restrict__ dst = w.out_ids + prefix;
  // Valid input gives every tile a disjoint byte range and at most one output
  // per byte, so prefix + cnt <= n.  Invalid input (whose output is discarded)
  // can break both; the bounds below keep even that inside the buffers.
  const uint32_t lim = prefix < w.n ? min(cnt, w.n - prefix) : 0u;
  for (uint32_t i = (uint32_t)tid; i < lim; i += EMIT_THREADS) {
    const uint32_t v = src[i];
    dst[i] = MODE == 1 ? (v < tb.n_ids ? tb.ext_id[v] : -1) : (int32_t)v;
  }
  if (t == w.n_tiles - 1 && tid == 0) {
    const uint64_t e = __hip_atomic_load(&w.ctrl->err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *w.out_len = (uint32_t)(e >> 32) == w.epoch ? -(int64_t)(uint32_t)e : (int64_t)(prefix + cnt);
  }
}

// Exclusive prefix of the tile counts, one block (requests of many tiles).
__global__ __launch_bounds__(1024) void tile_scan_kernel(Work w) {
  __shared__ uint32_t s_w[16];
  const int tid = (int)threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  uint32_t carry = 0;
  for (uint32_t b0 = 0; b0 < w.n_tiles; b0 += 1024) {
    const uint32_t i = b0 + (uint32_t)tid;
    const uint32_t v = i < w.n_tiles ? w.tile_cnt[i] : 0u;
    const uint32_t inc = wave_incl_sum(v, lane);
    if (lane == 63) s_w[wave] = inc;
    __syncthreads();
    uint32_t wpre = 0, tot = 0;
    for (int k = 0; k < 16; ++k) {
      if (k < wave) wpre += s_w[k];
      tot += s_w[k];
    }
    if (i < w.n_tiles) w.tile_pre[i] = carry + wpre + inc - v;
    carry += tot;
    __syncthreads();
  }
}

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

hipError_t launch_emit(const Work& w, const DevTables& tb, int mode, hipStream_t s) {
  const int direct = w.n_tiles <= EMIT_DIRECT_TILES ? 1 : 0;
  if (mode == 1)
    hipLaunchKernelGGL(emit_kernel<1>, dim3(w.n_tiles), dim3(EMIT_THREADS), 0, s, w, tb, direct);
  else
    hipLaunchKernelGGL(emit_kernel<0>, dim3(w.n_tiles), dim3(EMIT_THREADS), 0, s, w, tb, direct);
  return hipGetLastError();
}

hipError_t launch_tile_scan(const Work& w, hipStream_t s) {
  hipLaunchKernelGGL(tile_scan_kernel, dim3(1), dim3(1024), 0, s, w);
  return hipGetLastError();
}

hipError_t launch_doc_offsets(const Work& w, hipStream_t s) {
  uint32_t blocks = (uint32_t)((w.n_docs + 1 + 255) / 256);
  if (blocks > 1024) blocks = 1024;
  hipLaunchKernelGGL(doc_offsets_kernel, dim3(blocks), dim3(256), 0, s, w);
  return hipGetLastError();
}

}  // namespace tt
