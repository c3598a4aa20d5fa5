// Exact byte-level BPE over the pieces, on the GPU.
//
// Each piece is encoded on its own: start from the IDs of its bytes and
// repeatedly merge the adjacent pair with the lowest merge rank, leftmost
// first (the model stage of the front-end/model factorisation, Appendix,
// Definition d:frontend and Lemma l:homo).  Two facts license a parallel
// schedule (Sec. 4.2, "GPU BPE"): the minimum rank of a round names one pair,
// and merging all leftmost non-overlapping occurrences of that pair at once
// equals merging them one by one; and after a merge only the two pairs next
// to it need a new rank lookup.  Work is dispatched by piece length so each
// piece gets the smallest execution unit that holds it (Sec. 4.2).
//
// MI355X design (wave64, LDS, one HBM-resident hash table):
//   - pieces of at most 16 bytes: one thread per piece, the sequence in
//     registers; ranks come from the open-addressing merge table;
//   - 17..512 bytes: one 64-lane wave per piece, the sequence in LDS laid out
//     as rows of 64 tokens; a round is a wave min-reduction, one ballot per
//     row, a closed-form leftmost non-overlapping selection on the 64-bit
//     mask, a popcount compaction and the neighbour re-probes;
//   - longer pieces: the same rounds with 16 waves per piece and the rows in
//     global memory; pieces reach this engine through a device work queue.
// Pieces go to the wave and block engines through device-side queues, so no
// count is read back by the host.
#include "tt_internal.h"

namespace tt {

namespace {

constexpr uint32_t RANK_DIRTY = 0xFFFFFFFEu;  // pair changed; rank to be probed again

__device__ __forceinline__ uint32_t wave_min(uint32_t v) {
#pragma unroll
  for (int d = 32; d >= 1; d >>= 1) v = min(v, (uint32_t)__shfl_xor(v, d, 64));
  return v;
}

// Leftmost non-overlapping choice among the set bits of m, where bit j stands
// for the pair (token j, token j+1).  Within every run of consecutive set bits
// the greedy left-to-right choice takes the run's first bit and every second
// bit after it.  Runs that start on an even bit are isolated with one carry
// propagation: adding their start bits clears exactly those runs.
__device__ __forceinline__ uint64_t leftmost_nonoverlapping(uint64_t m) {
  const uint64_t EVEN = 0x5555555555555555ull;
  uint64_t starts = m & ~(m << 1);
  uint64_t even_runs = ((m + (starts & EVEN)) ^ m) & m;
  return (even_runs & EVEN) | (m & ~even_runs & ~EVEN);
}

__device__ __forceinline__ uint64_t lanemask_lt(int lane) {
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

}  // namespace

// ---------------------------------------------------------------------------
// Short pieces: one thread per piece.
//
// A piece of at most 16 bytes lives in 16 token slots.  Pair ranks stay in
// registers; token IDs and merge results live in LDS as [slot][thread], so the
// bank of an access depends only on the thread and per-thread slot indices
// never conflict.  A merge clears the right token's bit in an alive mask
// instead of shifting the tail; neighbours are found with bit scans.  The
// per-piece chain is one probe round trip for the initial pairs (issued four
// at a time) plus one per merge (its two re-probes overlap).
// ---------------------------------------------------------------------------
constexpr int SP_THREADS = 256;

__global__ __launch_bounds__(SP_THREADS) void bpe_small_kernel(Work w, DevTables tb) {
  __shared__ int32_t s_bid[256];
  __shared__ uint32_t s_ids[SMALL_MAX][SP_THREADS];
  __shared__ uint32_t s_res[SMALL_MAX][SP_THREADS];
  const int tid = threadIdx.x;
  s_bid[tid] = tb.byte_id[tid];
  __syncthreads();
  const uint32_t P = w.ctrl->n_pieces;
  const uint32_t stride = gridDim.x * blockDim.x;
  const MergeSlot* __restrict__ tab = tb.slots;
  const uint32_t mask = tb.mask;
  for (uint32_t p = blockIdx.x * blockDim.x + tid; p < P; p += stride) {
    const uint32_t a = w.piece_off[p];
    const uint32_t L = w.piece_off[p + 1] - a;
    if (L > (uint32_t)SMALL_MAX) {
      uint32_t k = atomicAdd(&w.ctrl->n_long, 1u);
      w.long_list[k] = p;
      continue;
    }
    uint32_t id0[SMALL_MAX];
#pragma unroll
    for (int j = 0; j < SMALL_MAX; ++j) {
      id0[j] = (uint32_t)j < L ? (uint32_t)s_bid[w.text[a + j]] : 0u;
      s_ids[j][tid] = id0[j];
    }
    uint32_t rk[SMALL_MAX];
#pragma unroll
    for (int g = 0; g < SMALL_MAX; g += 4) {
      uint32_t si[4];
      uint4 sv[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int j = g + k;
        if (j + 1 < SMALL_MAX && (uint32_t)(j + 1) < L) {
          si[k] = probe_start(mask, id0[j], id0[j + 1]);
          sv[k] = load_slot(tab, si[k]);
        }
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int j = g + k;
        uint2 r = make_uint2(RANK_INF, 0u);
        if (j + 1 < SMALL_MAX && (uint32_t)(j + 1) < L) r = probe_finish(tab, mask, si[k], sv[k], id0[j], id0[j + 1]);
        rk[j] = r.x;
        s_res[j][tid] = r.y;
      }
    }
    uint32_t alive = L >= 32 ? 0xFFFFFFFFu : ((1u << L) - 1u);
    for (;;) {
      uint32_t best = RANK_INF;
      int k = 0;
#pragma unroll
      for (int j = 0; j < SMALL_MAX - 1; ++j)
        if (rk[j] < best) {
          best = rk[j];
          k = j;
        }
      if (best == RANK_INF) break;
      // token k absorbs the next live token m
      const uint32_t above_k = alive & ~((2u << k) - 1u);
      const int m = __builtin_ctz(above_k);
      alive &= ~(1u << m);
      const uint32_t above_m = alive & ~((2u << m) - 1u);
      const uint32_t below_k = alive & ((1u << k) - 1u);
      const uint32_t nid = s_res[k][tid];
      s_ids[k][tid] = nid;
      const bool hr = above_m != 0, hl = below_k != 0;
      const int r_i = hr ? __builtin_ctz(above_m) : 0;
      const int l_i = hl ? 31 - __builtin_clz(below_k) : 0;
      const uint32_t right = s_ids[r_i][tid];
      const uint32_t left = s_ids[l_i][tid];
      uint32_t il = 0, ir = 0;
      uint4 sl = make_uint4(EMPTY, 0, 0, 0), sr = make_uint4(EMPTY, 0, 0, 0);
      if (hr) {
        ir = probe_start(mask, nid, right);
        sr = load_slot(tab, ir);
      }
      if (hl) {
        il = probe_start(mask, left, nid);
        sl = load_slot(tab, il);
      }
      uint2 rr = make_uint2(RANK_INF, 0u), rl = make_uint2(RANK_INF, 0u);
      if (hr) rr = probe_finish(tab, mask, ir, sr, nid, right);
      if (hl) rl = probe_finish(tab, mask, il, sl, left, nid);
      s_res[k][tid] = rr.y;
      if (hl) s_res[l_i][tid] = rl.y;
#pragma unroll
      for (int j = 0; j < SMALL_MAX; ++j) {
        if (j == m) rk[j] = RANK_INF;
        if (j == k) rk[j] = rr.x;
        if (hl && j == l_i) rk[j] = rl.x;
      }
    }
    int32_t* out = w.ids + a;
    uint32_t c = 0;
    for (uint32_t al = alive; al; al &= al - 1u) out[c++] = (int32_t)s_ids[__builtin_ctz(al)][tid];
    w.piece_cnt[p] = c;
  }
}

// ---------------------------------------------------------------------------
// Round engine over rows of 64 tokens, shared by the wave engine (NW = 1,
// rows in LDS) and the block engine (NW = 16, rows in global memory).
// ---------------------------------------------------------------------------
template <int NW>
struct RoundShared {
  uint32_t wmin[NW];
  uint32_t f0[NW], f1[NW], cin[NW];
  uint32_t wsum[NW], wbase[NW];
  uint32_t n_next;
};

template <int NW>
__device__ void bpe_rounds(uint32_t* ids0, uint32_t* ids1, uint32_t* rk0, uint32_t* rk1, uint32_t* rs0,
                           uint32_t* rs1, uint64_t* sel, const uint8_t* bytes, uint32_t L,
                           const int32_t* bid, const DevTables& tb, int32_t* out, uint32_t* out_cnt,
                           RoundShared<NW>& sm) {
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  constexpr int NT = NW * 64;
  uint32_t* ids[2] = {ids0, ids1};
  uint32_t* rk[2] = {rk0, rk1};
  uint32_t* rs[2] = {rs0, rs1};
  int cur = 0;
  uint32_t n = L;

  for (uint32_t i = tid; i < n; i += NT) ids[0][i] = (uint32_t)bid[bytes[i]];
  __syncthreads();
  for (uint32_t i = tid; i < n; i += NT) {
    uint2 r = make_uint2(RANK_INF, 0u);
    if (i + 1 < n) r = probe_pair(tb.slots, tb.mask, ids[0][i], ids[0][i + 1]);
    rk[0][i] = r.x;
    rs[0][i] = r.y;
  }
  __syncthreads();

  for (;;) {
    const uint32_t* I = ids[cur];
    const uint32_t* R = rk[cur];
    const uint32_t* S = rs[cur];
    uint32_t* I2 = ids[cur ^ 1];
    uint32_t* R2 = rk[cur ^ 1];
    uint32_t* S2 = rs[cur ^ 1];

    // 1. lowest rank in the piece
    uint32_t m = RANK_INF;
    for (uint32_t i = tid; i < n; i += NT) m = min(m, R[i]);
    m = wave_min(m);
    if (NW > 1) {
      if (lane == 0) sm.wmin[wave] = m;
      __syncthreads();
      m = RANK_INF;
      for (int v = 0; v < NW; ++v) m = min(m, sm.wmin[v]);
    }
    if (m == RANK_INF) break;

    // 2. leftmost non-overlapping occurrences, row by row.  A row's choice
    // depends on whether the last pair of the previous row was chosen; with
    // several waves each wave first evaluates its rows for both carries.
    const uint32_t rows = (n + 63) / 64;
    const uint32_t rpw = (rows + NW - 1) / NW;
    const uint32_t r_lo = min(rows, (uint32_t)wave * rpw);
    const uint32_t r_hi = min(rows, r_lo + rpw);
    uint32_t carry = 0;
    if (NW > 1) {
      uint32_t c0 = 0, c1 = 1;
      for (uint32_t r = r_lo; r < r_hi; ++r) {
        uint32_t i = r * 64 + lane;
        uint64_t occ = __ballot(i < n && R[i] == m);
        c0 = (uint32_t)(leftmost_nonoverlapping(occ & ~(uint64_t)c0) >> 63);
        c1 = (uint32_t)(leftmost_nonoverlapping(occ & ~(uint64_t)c1) >> 63);
      }
      if (lane == 0) {
        sm.f0[wave] = c0;
        sm.f1[wave] = c1;
      }
      __syncthreads();
      if (tid == 0) {
        uint32_t c = 0;
        for (int v = 0; v < NW; ++v) {
          sm.cin[v] = c;
          c = c ? sm.f1[v] : sm.f0[v];
        }
      }
      __syncthreads();
      carry = sm.cin[wave];
    }
    uint32_t keep_total = 0;
    for (uint32_t r = r_lo; r < r_hi; ++r) {
      uint32_t i = r * 64 + lane;
      uint64_t occ = __ballot(i < n && R[i] == m);
      uint64_t s = leftmost_nonoverlapping(occ & ~(uint64_t)carry);
      if (lane == 0) sel[r] = s;
      uint64_t valid = (n - r * 64 >= 64) ? ~0ull : ((1ull << (n - r * 64)) - 1ull);
      uint64_t keep = valid & ~((s << 1) | (uint64_t)carry);
      keep_total += __popcll(keep);
      carry = (uint32_t)(s >> 63);
    }
    if (lane == 0) sel[rows] = 0;  // sentinel row (only bit 0 is ever read)
    // 3. compaction offsets
    if (NW > 1) {
      if (lane == 0) sm.wsum[wave] = keep_total;
      __syncthreads();
      if (tid == 0) {
        uint32_t b = 0;
        for (int v = 0; v < NW; ++v) {
          sm.wbase[v] = b;
          b += sm.wsum[v];
        }
        sm.n_next = b;
      }
      __syncthreads();
    } else {
      __syncthreads();
    }
    uint32_t base = NW > 1 ? sm.wbase[wave] : 0u;
    const uint32_t n2 = NW > 1 ? sm.n_next : keep_total;
    uint32_t prevbit = (NW > 1 && r_lo > 0) ? (uint32_t)(sel[r_lo - 1] >> 63) : 0u;
    for (uint32_t r = r_lo; r < r_hi; ++r) {
      uint32_t i = r * 64 + lane;
      uint64_t s = sel[r];
      uint64_t valid = (n - r * 64 >= 64) ? ~0ull : ((1ull << (n - r * 64)) - 1ull);
      uint64_t keep = valid & ~((s << 1) | (uint64_t)prevbit);
      if ((keep >> lane) & 1ull) {
        uint32_t k = base + __popcll(keep & lanemask_lt(lane));
        uint32_t my = (uint32_t)(s >> lane) & 1u;
        uint32_t nx = lane < 63 ? (uint32_t)(s >> (lane + 1)) & 1u : (uint32_t)(sel[r + 1] & 1ull);
        I2[k] = my ? S[i] : I[i];
        R2[k] = (my | nx) ? RANK_DIRTY : R[i];
        S2[k] = S[i];
      }
      base += __popcll(keep);
      prevbit = (uint32_t)(s >> 63);
    }
    __syncthreads();
    n = n2;
    // 4. ranks of the pairs next to the merges
    for (uint32_t i = tid; i < n; i += NT) {
      if (R2[i] == RANK_DIRTY) {
        uint2 r = make_uint2(RANK_INF, 0u);
        if (i + 1 < n) r = probe_pair(tb.slots, tb.mask, I2[i], I2[i + 1]);
        R2[i] = r.x;
        S2[i] = r.y;
      }
    }
    __syncthreads();
    cur ^= 1;
  }
  const uint32_t* I = ids[cur];
  for (uint32_t i = tid; i < n; i += NT) out[i] = (int32_t)I[i];
  if (tid == 0) *out_cnt = n;
}

// ---------------------------------------------------------------------------
// Wave engine: one 64-thread block pulls pieces from the queue.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void bpe_wave_kernel(Work w, DevTables tb) {
  __shared__ uint32_t s_ids[2][WAVE_MAX], s_rk[2][WAVE_MAX], s_rs[2][WAVE_MAX];
  __shared__ uint64_t s_sel[WAVE_MAX / 64 + 1];
  __shared__ int32_t s_bid[256];
  __shared__ RoundShared<1> sm;
  for (int i = threadIdx.x; i < 256; i += 64) s_bid[i] = tb.byte_id[i];
  __syncthreads();
  const uint32_t n_long = w.ctrl->n_long;
  for (;;) {
    uint32_t k = 0;
    if (threadIdx.x == 0) k = atomicAdd(&w.ctrl->long_ticket, 1u);
    k = __shfl(k, 0, 64);
    if (k >= n_long) break;
    const uint32_t p = w.long_list[k];
    const uint32_t a = w.piece_off[p];
    const uint32_t L = w.piece_off[p + 1] - a;
    if (L > (uint32_t)WAVE_MAX) {
      if (threadIdx.x == 0) {
        uint32_t z = atomicAdd(&w.ctrl->n_big, 1u);
        w.big_list[z] = p;
      }
      continue;
    }
    bpe_rounds<1>(s_ids[0], s_ids[1], s_rk[0], s_rk[1], s_rs[0], s_rs[1], s_sel, w.text + a, L, s_bid, tb,
                  w.ids + a, w.piece_cnt + p, sm);
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Block engine: 16 waves per piece, rows in global scratch.
// ---------------------------------------------------------------------------
constexpr int BIG_WAVES = 16;

__global__ __launch_bounds__(BIG_WAVES * 64) void bpe_big_kernel(Work w, DevTables tb) {
  __shared__ int32_t s_bid[256];
  __shared__ RoundShared<BIG_WAVES> sm;
  __shared__ uint32_t s_k;
  for (int i = threadIdx.x; i < 256; i += blockDim.x) s_bid[i] = tb.byte_id[i];
  __syncthreads();
  const uint32_t n_big = w.ctrl->n_big;
  const uint32_t n = w.n;
  for (;;) {
    if (threadIdx.x == 0) s_k = atomicAdd(&w.ctrl->big_ticket, 1u);
    __syncthreads();
    const uint32_t k = s_k;
    __syncthreads();
    if (k >= n_big) break;
    const uint32_t p = w.big_list[k];
    const uint32_t a = w.piece_off[p];
    const uint32_t L = w.piece_off[p + 1] - a;
    uint32_t* sc = w.scratch32;
    uint64_t* sel = reinterpret_cast<uint64_t*>(sc + 6ull * n) + a / 32;
    bpe_rounds<BIG_WAVES>(sc + a, sc + n + a, sc + 2ull * n + a, sc + 3ull * n + a, sc + 4ull * n + a,
                          sc + 5ull * n + a, sel, w.text + a, L, s_bid, tb, w.ids + a, w.piece_cnt + p, sm);
    __syncthreads();
  }
}

// Geometry depends only on the request size, never on counts the host would
// have to read back: the kernels read P and the queue lengths on the device.
hipError_t launch_bpe_small(const Work& w, const DevTables& t, hipStream_t s) {
  uint32_t est = w.n / 4 + 1;  // one thread per piece slot (P <= n), grid-stride beyond
  uint32_t blocks = (est + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  hipLaunchKernelGGL(bpe_small_kernel, dim3(blocks), dim3(256), 0, s, w, t);
  return hipGetLastError();
}

hipError_t launch_bpe_wave(const Work& w, const DevTables& t, hipStream_t s) {
  uint32_t blocks = w.n / 64 + 1;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(bpe_wave_kernel, dim3(blocks), dim3(64), 0, s, w, t);
  return hipGetLastError();
}

hipError_t launch_bpe_block(const Work& w, const DevTables& t, hipStream_t s) {
  uint32_t blocks = w.n / 4096 + 1;
  if (blocks > 256) blocks = 256;
  hipLaunchKernelGGL(bpe_big_kernel, dim3(blocks), dim3(BIG_WAVES * 64), 0, s, w, t);
  return hipGetLastError();
}

}  // namespace tt
