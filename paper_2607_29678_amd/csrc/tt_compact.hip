// Output compaction: scatter the per-piece IDs into one dense array.
//
// The BPE engines leave piece p's IDs at its byte offset and its token count
// in piece_cnt[p].  An exclusive scan of the counts gives every piece its
// output offset; the IDs are then copied (Sec. 4.2: the complete path is
// pre-tokenization, BPE and output compaction).  One pass: a block scan plus
// a decoupled look-back over the per-block totals.  The output length stays
// in device memory (Sec. 4.3: piece counts, dispatch lists and output length
// stay on the device).
#include "tt_internal.h"

namespace tt {

namespace {
constexpr uint32_t ST_AGG = 1u, ST_INC = 2u;
constexpr uint32_t LONG_COPY = 32;  // pieces with more IDs are copied by the whole block
}  // namespace

__global__ __launch_bounds__(CT_THREADS) void compact_kernel(Work w) {
  __shared__ uint32_t s_tile, s_prefix, s_nlong;
  __shared__ uint32_t s_wave[CT_THREADS / 64];
  __shared__ uint32_t s_long_p[CT_TILE], s_long_o[CT_TILE];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const uint32_t P = w.ctrl->n_pieces;
  const uint32_t n_tiles = (P + CT_TILE - 1) / CT_TILE;
  if (tid == 0) {
    s_tile = atomicAdd(&w.ctrl->ctile_ticket, 1u);
    s_nlong = 0;
  }
  __syncthreads();
  const uint32_t t = s_tile;
  if (P == 0) {
    // no character at all (only possible for invalid input): still report
    if (t == 0 && tid == 0) {
      w.piece_out[0] = 0;
      uint32_t err = __hip_atomic_load(&w.ctrl->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      int64_t len = err ? -(int64_t)err : 0;
      w.ctrl->out_len = len;
      if (w.out_len) *w.out_len = len;
    }
    return;
  }
  if (t >= n_tiles) return;
  const uint32_t p0 = t * CT_TILE + tid * CT_PPT;
  uint32_t c[CT_PPT];
  uint32_t mine = 0;
#pragma unroll
  for (int j = 0; j < CT_PPT; ++j) {
    uint32_t p = p0 + j;
    c[j] = p < P ? w.piece_cnt[p] : 0u;
    mine += c[j];
  }
  uint32_t inc = mine;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    uint32_t o = __shfl_up(inc, d, 64);
    if (lane >= d) inc += o;
  }
  if (lane == 63) s_wave[wave] = inc;
  __syncthreads();
  uint32_t wpre = 0, total = 0;
  for (int v = 0; v < CT_THREADS / 64; ++v) {
    if (v < wave) wpre += s_wave[v];
    total += s_wave[v];
  }
  const uint32_t texcl = wpre + inc - mine;
  if (wave == 0) {
    if (lane == 0)
      __hip_atomic_store(&w.ctile_status[t], ((uint64_t)ST_AGG << 32) | total, __ATOMIC_RELEASE,
                         __HIP_MEMORY_SCOPE_AGENT);
    uint32_t prefix = 0;
    for (int64_t base = (int64_t)t - 1; base >= 0; base -= 64) {
      int64_t j = base - lane;
      uint64_t v = 0;
      if (j >= 0) {
        do {
          v = __hip_atomic_load(&w.ctile_status[j], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
        } while ((v >> 32) == 0);
      }
      bool incl = j < 0 || (v >> 32) == ST_INC;
      uint64_t m = __ballot(incl);
      int first = m ? (__ffsll((unsigned long long)m) - 1) : 64;
      uint32_t x = (j >= 0 && lane <= first) ? (uint32_t)v : 0u;
#pragma unroll
      for (int d = 32; d >= 1; d >>= 1) x += __shfl_xor(x, d, 64);
      prefix += x;
      if (m) break;
    }
    if (lane == 0) {
      __hip_atomic_store(&w.ctile_status[t], ((uint64_t)ST_INC << 32) | (prefix + total), __ATOMIC_RELEASE,
                         __HIP_MEMORY_SCOPE_AGENT);
      s_prefix = prefix;
    }
  }
  __syncthreads();
  uint32_t o = s_prefix + texcl;
#pragma unroll
  for (int j = 0; j < CT_PPT; ++j) {
    uint32_t p = p0 + j;
    if (p < P) {
      w.piece_out[p] = o;
      if (c[j] > LONG_COPY) {
        uint32_t k = atomicAdd(&s_nlong, 1u);
        s_long_p[k] = p;
        s_long_o[k] = o;
      } else {
        const int32_t* src = w.ids + w.piece_off[p];
        for (uint32_t i = 0; i < c[j]; ++i) w.out_ids[o + i] = src[i];
      }
    }
    o += c[j];
  }
  __syncthreads();
  for (uint32_t k = 0; k < s_nlong; ++k) {
    uint32_t p = s_long_p[k], ob = s_long_o[k];
    const int32_t* src = w.ids + w.piece_off[p];
    uint32_t cnt = w.piece_cnt[p];
    for (uint32_t i = tid; i < cnt; i += CT_THREADS) w.out_ids[ob + i] = src[i];
  }
  if (t == n_tiles - 1 && tid == 0) {
    uint32_t T = s_prefix + total;
    w.piece_out[P] = T;
    uint32_t err = __hip_atomic_load(&w.ctrl->error, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    int64_t len = err ? -(int64_t)err : (int64_t)T;
    w.ctrl->out_len = len;
    if (w.out_len) *w.out_len = len;
  }
}

hipError_t launch_compact(const Work& w, uint32_t n_ct_tiles, hipStream_t s) {
  hipLaunchKernelGGL(compact_kernel, dim3(n_ct_tiles), dim3(CT_THREADS), 0, s, w);
  return hipGetLastError();
}

// Batch: output offset of every document = output offset of its first piece.
__global__ void doc_offsets_kernel(Work w) {
  const uint32_t P = w.ctrl->n_pieces;
  for (int j = blockIdx.x * blockDim.x + threadIdx.x; j <= w.n_docs; j += gridDim.x * blockDim.x) {
    uint32_t d = (uint32_t)w.doc_off[j];
    uint32_t lo = 0, hi = P;  // first piece starting at or after d
    while (lo < hi) {
      uint32_t mid = (lo + hi) >> 1;
      if (w.piece_off[mid] < d) lo = mid + 1;
      else hi = mid;
    }
    w.out_doc_off[j] = (int64_t)w.piece_out[lo];
  }
}

hipError_t launch_doc_offsets(const Work& w, hipStream_t s) {
  int blocks = (w.n_docs + 1 + 255) / 256;
  hipLaunchKernelGGL(doc_offsets_kernel, dim3(blocks), dim3(256), 0, s, w);
  return hipGetLastError();
}

}  // namespace tt
