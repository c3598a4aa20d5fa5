// Exact byte-level BPE of one unit (a piece, or a segment of a piece that no
// merge can cross), on the GPU.
//
// A unit starts as the IDs of its bytes; the adjacent pair with the lowest
// merge rank is merged, leftmost first, until no pair has a rank (the model
// stage of the front-end/model factorisation, Appendix, Definition
// d:frontend and Lemma l:homo).  Two facts license the parallel schedules
// below (Sec. 4.2, "GPU BPE"): with a proper merge list, merging all leftmost
// non-overlapping occurrences of the round's lowest-ranked pair at once equals
// merging them one by one, and after a merge only the pairs that touch the new
// token need a new rank lookup.  The unit length picks the execution unit
// (Sec. 4.2 dispatches by piece length):
//   bpe_thread  <= 16 bytes: one thread, the unit in registers;
//   bpe_wave    <= 64 bytes: one wave64, one token per lane;
//   bpe_pair32  two units of <= 32 bytes: one wave64, one unit per half;
//   bpe_rows    longer:      NW waves over rows of 64 tokens in LDS or global
//                            memory.
// IDs are internal: byte b is b, the result of merge r is 256 + r.
#pragma once

#include "tt_internal.h"

namespace tt {

constexpr uint32_t RANK_DIRTY = 0xFFFFFFFEu;  // pair changed; its rank must be looked up again

// Leftmost non-overlapping choice among the set bits of m, where bit j stands
// for the pair (token j, token j+1).  Two chosen pairs may not share a token,
// so within every run of consecutive set bits the left-to-right greedy choice
// takes the run's first bit and every second bit after it.  Runs that start on
// an even bit are isolated with one carry propagation: adding their start bits
// clears exactly those runs.
__device__ __forceinline__ uint64_t leftmost_nonoverlapping(uint64_t m) {
  const uint64_t EVEN = 0x5555555555555555ull;
  const uint64_t starts = m & ~(m << 1);
  const uint64_t even_runs = ((m + (starts & EVEN)) ^ m) & m;
  return (even_runs & EVEN) | (m & ~even_runs & ~EVEN);
}

// Number of set bits of m below the calling lane.
__device__ __forceinline__ uint32_t bits_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// Minimum over the 64 lanes of a wave, in every lane (DPP row steps, then
// the row broadcasts; the full result ends in lane 63).
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
  int x = (int)v;
  x = (int)min((uint32_t)x, (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  x = (int)min((uint32_t)x, (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  x = (int)min((uint32_t)x, (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0x141, 0xF, 0xF, false));  // row_half_mirror
  x = (int)min((uint32_t)x, (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0x140, 0xF, 0xF, false));  // row_mirror
  x = (int)min((uint32_t)x, (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0x142, 0xA, 0xF, false));  // row_bcast15
  x = (int)min((uint32_t)x, (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0x143, 0xC, 0xF, false));  // row_bcast31
  return (uint32_t)__builtin_amdgcn_readlane(x, 63);
}

// Inclusive sum over the lanes of a wave (DPP: shifts within rows of 16
// lanes, then the row broadcasts carry row totals forward).
__device__ __forceinline__ uint32_t wave_incl_sum(uint32_t v) {
  int x = (int)v;
  x += __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);  // row_shr:1
  x += __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);  // row_shr:2
  x += __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, true);  // row_shr:4
  x += __builtin_amdgcn_update_dpp(0, x, 0x118, 0xF, 0xF, true);  // row_shr:8
  x += __builtin_amdgcn_update_dpp(0, x, 0x142, 0xA, 0xF, false); // row_bcast:15 into rows 1, 3
  x += __builtin_amdgcn_update_dpp(0, x, 0x143, 0xC, 0xF, false); // row_bcast:31 into rows 2, 3
  return (uint32_t)x;
}

// ---------------------------------------------------------------------------
// One thread, at most 16 bytes.  The unit's tokens live in its own LDS words
// ids[0..L) (the caller puts the bytes there; merged tokens overwrite their
// left operand in place, and the tokens end compacted in ids[0..count)).  The
// rank of the pair at slot j is kept in LDS at rk[j * TH_THREADS]: the caller
// passes its own column of a [SMALL_MAX - 1][TH_THREADS] array (the last slot
// never has a pair), so the lanes of a wave never share a bank.  A rank is
// kept as (rank << 4) | j, so that one unsigned minimum finds the lowest rank
// and, among equal ranks (the same pair), the leftmost occurrence; a merge
// rewrites at most three slots with three stores.  A merge clears the right
// token's bit in an alive mask instead of shifting the tail.  The chain is one
// round trip for the initial byte pairs (all loads in flight at once) and one
// per merge (its two neighbour lookups overlap).  Returns the number of tokens.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t bpe_thread(uint32_t L, uint32_t* ids, uint32_t* rk, const DevTables& tb) {
  constexpr int S = SMALL_MAX;
  constexpr int ST = TH_THREADS;
  const u64x2* __restrict__ tab = tb.slots;
  const uint32_t nb = tb.nb;
  {
    uint32_t b[S], r[S - 1];
#pragma unroll
    for (int j = 0; j < S; ++j) b[j] = (uint32_t)j < L ? ids[j] : 0u;
    // every initial rank load is issued before any is used (no branches)
#pragma unroll
    for (int j = 0; j < S - 1; ++j) r[j] = tb.pair0[(b[j] << 8) | b[j + 1]];
#pragma unroll
    for (int j = 0; j < S - 1; ++j)
      rk[j * ST] = ((uint32_t)(j + 1) < L && r[j] != RANK_INF) ? ((r[j] << 4) | (uint32_t)j) : RANK_INF;
  }
  uint32_t alive = (1u << L) - 1u;  // L <= 16
  for (;;) {
    uint32_t best = RANK_INF;
#pragma unroll
    for (int j = 0; j < S - 1; ++j) best = min(best, rk[j * ST]);
    if (best == RANK_INF) break;
    const uint32_t k = best & 15u;
    const uint32_t nid = 256u + (best >> 4);
    // token k absorbs the next live token m
    const uint32_t m = (uint32_t)__builtin_ctz(alive & ~((2u << k) - 1u));
    alive &= ~(1u << m);
    const uint32_t above_m = alive & ~((2u << m) - 1u);
    const uint32_t below_k = alive & ((1u << k) - 1u);
    const bool hr = above_m != 0u, hl = below_k != 0u;
    const uint32_t right = ids[hr ? (uint32_t)__builtin_ctz(above_m) : k];
    const uint32_t l_i = hl ? 31u - (uint32_t)__builtin_clz(below_k) : k;
    const uint32_t left = ids[l_i];
    ids[k] = nid;
    // both lookups are issued unconditionally (a missing neighbour looks up a
    // harmless pair) so that their four loads are in flight together
    const ProbeIssued pr = probe_issue(tab, nb, nid, right);
    const ProbeIssued pl = probe_issue(tab, nb, left, nid);
    const uint32_t rr = hr ? probe_finish(pr, nid, right) : RANK_INF;
    const uint32_t rl = probe_finish(pl, left, nid);
    if (m < (uint32_t)(S - 1)) rk[m * ST] = RANK_INF;
    rk[k * ST] = rr == RANK_INF ? RANK_INF : ((rr << 4) | k);
    if (hl) rk[l_i * ST] = rl == RANK_INF ? RANK_INF : ((rl << 4) | l_i);
  }
  // compact in place: the c-th live token moves to ids[c], c <= its slot
  uint32_t c = 0;
  for (uint32_t al = alive; al; al &= al - 1u) ids[c++] = ids[__builtin_ctz(al)];
  return c;
}

// ---------------------------------------------------------------------------
// One wave64, at most 64 bytes: lane i holds token i and the rank of the pair
// (i, i+1).  A round is a wave minimum, one ballot, the closed-form leftmost
// non-overlapping choice, a push permute that compacts the survivors, and the
// rank lookups of the changed pairs (one probe round trip).  Every lane of the
// wave calls it with the same arguments.
// ---------------------------------------------------------------------------
template <class ByteF, class OutF>
__device__ __forceinline__ uint32_t bpe_wave(uint32_t L, ByteF byte, const DevTables& tb, OutF out) {
  const int lane = (int)(threadIdx.x & 63u);
  uint32_t n = L;  // <= 64
  uint32_t id = (uint32_t)lane < n ? byte(lane) : 0u;
  uint32_t idn = (uint32_t)__shfl_down((int)id, 1, 64);
  uint32_t rk = (uint32_t)lane + 1u < n ? tb.pair0[(id << 8) | idn] : RANK_INF;
  for (;;) {
    const uint32_t m = wave_min_u32(rk);
    if (m == RANK_INF) break;
    const uint64_t sel = leftmost_nonoverlapping(__ballot(rk == m));
    const uint64_t valid = n >= 64u ? ~0ull : ((1ull << n) - 1ull);
    const uint64_t keep = valid & ~(sel << 1);
    const bool me_sel = (sel >> lane) & 1ull;
    const bool nx_sel = lane < 63 && ((sel >> (lane + 1)) & 1ull);
    const uint32_t nid = me_sel ? 256u + m : id;
    const uint32_t r = (me_sel || nx_sel) ? RANK_DIRTY : rk;
    // at least one pair merged, so at most 63 tokens survive and lane 63 is
    // free to take the values of the lanes that do not survive
    const int dest = ((keep >> lane) & 1ull) ? (int)bits_below(keep) : 63;
    id = (uint32_t)__builtin_amdgcn_ds_permute(dest << 2, (int)nid);
    const uint32_t r2 = (uint32_t)__builtin_amdgcn_ds_permute(dest << 2, (int)r);
    n = (uint32_t)__popcll(keep);
    idn = (uint32_t)__shfl_down((int)id, 1, 64);
    rk = RANK_INF;
    if ((uint32_t)lane < n) {
      rk = r2;
      if (r2 == RANK_DIRTY) rk = (uint32_t)lane + 1u < n ? probe_rank(tb.slots, tb.nb, id, idn) : RANK_INF;
    }
  }
  if ((uint32_t)lane < n) out(lane, id);
  return n;
}

// ---------------------------------------------------------------------------
// Two units of at most 32 bytes on one wave64: lanes 0..31 hold the tokens of
// unit A, lanes 32..63 those of unit B, and each half runs the rounds of
// bpe_wave on its own unit (its own minimum, occurrences and compaction) until
// both are done; a half whose unit is done keeps its lanes in place.  The pair
// (lane 31, lane 32) is never a pair: the rank at lane 31 is always RANK_INF.
// byte(h, j) and out(h, j, id) take the half (0: A, 1: B) and the position in
// it.  Returns count(A) | count(B) << 16.  Every lane of the wave calls it
// with the same arguments.
// ---------------------------------------------------------------------------
// Minimum over the calling lane's half (32 lanes) of a wave: complete in
// lanes 31 and 63 (the row steps of wave_min_u32, then one row broadcast
// into rows 1 and 3).
__device__ __forceinline__ uint32_t half_min_u32(uint32_t v) {
  int x = (int)v;
  x = (int)min((uint32_t)x, (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0xB1, 0xF, 0xF, false));   // quad_perm 1,0,3,2
  x = (int)min((uint32_t)x, (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0x4E, 0xF, 0xF, false));   // quad_perm 2,3,0,1
  x = (int)min((uint32_t)x, (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0x141, 0xF, 0xF, false));  // row_half_mirror
  x = (int)min((uint32_t)x, (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0x140, 0xF, 0xF, false));  // row_mirror
  x = (int)min((uint32_t)x, (uint32_t)__builtin_amdgcn_update_dpp(x, x, 0x142, 0xA, 0xF, false));  // row_bcast15 into rows 1, 3
  return (uint32_t)x;
}

template <class ByteF, class OutF>
__device__ __forceinline__ uint32_t bpe_pair32(uint32_t LA, uint32_t LB, ByteF byte, const DevTables& tb, OutF out) {
  const int lane = (int)(threadIdx.x & 63u);
  const uint32_t h = (uint32_t)lane >> 5;  // 0: unit A, 1: unit B
  const uint32_t j = (uint32_t)lane & 31u;  // position in the half
  const uint64_t half = h ? 0xFFFFFFFF00000000ull : 0x00000000FFFFFFFFull;
  uint32_t n = h ? LB : LA;  // tokens of this half's unit (<= 32)
  uint32_t id = j < n ? byte(h, j) : 0u;
  uint32_t idn = (uint32_t)__shfl_down((int)id, 1, 64);
  uint32_t rk = j + 1u < n ? tb.pair0[(id << 8) | idn] : RANK_INF;
  for (;;) {
    const uint32_t mh = half_min_u32(rk);
    const uint32_t mA = (uint32_t)__builtin_amdgcn_readlane((int)mh, 31);
    const uint32_t mB = (uint32_t)__builtin_amdgcn_readlane((int)mh, 63);
    if (mA == RANK_INF && mB == RANK_INF) break;
    const uint32_t m = h ? mB : mA;
    const bool active = m != RANK_INF;  // this half merges this round
    const uint64_t sel = leftmost_nonoverlapping(__ballot(active && rk == m));
    const uint64_t keep = __ballot(j < n) & ~(sel << 1);
    const bool me_sel = (sel >> lane) & 1ull;
    const bool nx_sel = j < 31u && ((sel >> (lane + 1)) & 1ull);
    const uint32_t nid = me_sel ? 256u + m : id;
    const uint32_t r = (me_sel || nx_sel) ? RANK_DIRTY : rk;
    // a half that merged at least one pair has a free last lane for the
    // lanes that do not survive; a half that merged none stays in place
    const bool kept = (keep >> lane) & 1ull;
    const int dest = kept ? (int)(32u * h + bits_below(keep & half)) : active ? (int)(32u * h + 31u) : lane;
    id = (uint32_t)__builtin_amdgcn_ds_permute(dest << 2, (int)nid);
    const uint32_t r2 = (uint32_t)__builtin_amdgcn_ds_permute(dest << 2, (int)r);
    n = (uint32_t)__popcll(keep & half);
    idn = (uint32_t)__shfl_down((int)id, 1, 64);
    rk = RANK_INF;
    if (j < n) {
      rk = r2;
      if (r2 == RANK_DIRTY) rk = j + 1u < n ? probe_rank(tb.slots, tb.nb, id, idn) : RANK_INF;
    }
  }
  if (j < n) out(h, j, id);
  const uint32_t cA = (uint32_t)__builtin_amdgcn_readlane((int)n, 0);
  const uint32_t cB = (uint32_t)__builtin_amdgcn_readlane((int)n, 32);
  return cA | (cB << 16);
}

// ---------------------------------------------------------------------------
// One wave64, at most 128 bytes: lane i holds tokens i and 64 + i and the
// ranks of the pairs starting there.  A round is the same as in bpe_wave over
// a 128-bit occurrence mask (the choice in the second row continues the
// alternation of a run that crosses from the first, through the carry of the
// first row's last bit); the survivors are compacted through the wave's own
// 256 words of LDS `scr` (token IDs, then ranks), written and read back by the
// same wave.  Every lane of the wave calls it with the same arguments.
// ---------------------------------------------------------------------------
template <class ByteF, class OutF>
__device__ __forceinline__ uint32_t bpe_wave2(uint32_t L, ByteF byte, const DevTables& tb, uint32_t* scr, OutF out) {
  const int lane = (int)(threadIdx.x & 63u);
  const uint32_t l0 = (uint32_t)lane, l1 = 64u + (uint32_t)lane;
  uint32_t n = L;  // <= 128
  uint32_t id0 = l0 < n ? byte(lane) : 0u;
  uint32_t id1 = l1 < n ? byte(64 + lane) : 0u;
  auto next0 = [&]() -> uint32_t {  // token after position lane (row 0)
    const uint32_t nx = (uint32_t)__shfl_down((int)id0, 1, 64);
    const uint32_t head1 = (uint32_t)__builtin_amdgcn_readlane((int)id1, 0);
    return lane == 63 ? head1 : nx;
  };
  uint32_t nx0 = next0(), nx1 = (uint32_t)__shfl_down((int)id1, 1, 64);
  uint32_t rk0 = l0 + 1u < n ? tb.pair0[(id0 << 8) | nx0] : RANK_INF;
  uint32_t rk1 = l1 + 1u < n ? tb.pair0[(id1 << 8) | nx1] : RANK_INF;
  for (;;) {
    const uint32_t m = wave_min_u32(min(rk0, rk1));
    if (m == RANK_INF) break;
    const uint64_t s0 = leftmost_nonoverlapping(__ballot(rk0 == m));
    const uint64_t c = s0 >> 63;  // the pair (63, 64) is chosen: token 64 is taken
    const uint64_t s1 = leftmost_nonoverlapping(__ballot(rk1 == m) & ~c);
    const uint64_t v0 = n >= 64u ? ~0ull : ((1ull << n) - 1ull);
    const uint64_t v1 = n >= 128u ? ~0ull : (n > 64u ? ((1ull << (n - 64u)) - 1ull) : 0ull);
    const uint64_t k0 = v0 & ~(s0 << 1), k1 = v1 & ~((s1 << 1) | c);
    const bool me0 = (s0 >> lane) & 1ull, me1 = (s1 >> lane) & 1ull;
    const bool nxs0 = lane < 63 ? ((s0 >> (lane + 1)) & 1ull) != 0ull : (s1 & 1ull) != 0ull;
    const bool nxs1 = lane < 63 && ((s1 >> (lane + 1)) & 1ull) != 0ull;
    const uint32_t c0 = (uint32_t)__popcll(k0);
    if ((k0 >> lane) & 1ull) {
      const uint32_t p = bits_below(k0);
      scr[p] = me0 ? 256u + m : id0;
      scr[128 + p] = (me0 || nxs0) ? RANK_DIRTY : rk0;
    }
    if ((k1 >> lane) & 1ull) {
      const uint32_t p = c0 + bits_below(k1);
      scr[p] = me1 ? 256u + m : id1;
      scr[128 + p] = (me1 || nxs1) ? RANK_DIRTY : rk1;
    }
    n = c0 + (uint32_t)__popcll(k1);
    // (one wave writes and reads its own words: LDS operations of a wave are
    // performed in order)
    id0 = l0 < n ? scr[l0] : 0u;
    const uint32_t r0 = l0 < n ? scr[128 + l0] : RANK_INF;
    id1 = l1 < n ? scr[l1] : 0u;
    const uint32_t r1 = l1 < n ? scr[128 + l1] : RANK_INF;
    nx0 = next0();
    nx1 = (uint32_t)__shfl_down((int)id1, 1, 64);
    rk0 = r0;
    if (r0 == RANK_DIRTY) rk0 = l0 + 1u < n ? probe_rank(tb.slots, tb.nb, id0, nx0) : RANK_INF;
    rk1 = r1;
    if (r1 == RANK_DIRTY) rk1 = l1 + 1u < n ? probe_rank(tb.slots, tb.nb, id1, nx1) : RANK_INF;
  }
  if (l0 < n) out(lane, id0);
  if (l1 < n) out(64 + lane, id1);
  return n;
}

// ---------------------------------------------------------------------------
// NW waves over rows of 64 tokens.  I0/I1 (IDs) and R0/R1 (pair ranks) are
// double buffers of at least L words, `sel` holds rows(L) + 1 selection masks;
// they may live in LDS or in global memory (visible to the whole block).
// Every thread of the block calls it with the same arguments.
// ---------------------------------------------------------------------------
template <int NW>
struct RowsShared {
  uint32_t wmin[NW];
  uint32_t f0[NW], f1[NW], cin[NW];
  uint32_t wsum[NW], wbase[NW];
  uint32_t n_next;
};

template <int NW, class ByteF, class OutF>
__device__ uint32_t bpe_rows(uint32_t L, ByteF byte, const DevTables& tb, uint32_t* I0, uint32_t* I1, uint32_t* R0,
                             uint32_t* R1, uint64_t* sel, RowsShared<NW>& sm, OutF out) {
  const int tid = (int)threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  constexpr int NT = NW * 64;
  uint32_t* ids[2] = {I0, I1};
  uint32_t* rk[2] = {R0, R1};
  int cur = 0;
  uint32_t n = L;

  for (uint32_t i = tid; i < n; i += NT) I0[i] = byte(i);
  __syncthreads();
  for (uint32_t i = tid; i < n; i += NT) R0[i] = i + 1 < n ? tb.pair0[(I0[i] << 8) | I0[i + 1]] : RANK_INF;
  __syncthreads();

  for (;;) {
    const uint32_t* I = ids[cur];
    const uint32_t* R = rk[cur];
    uint32_t* I2 = ids[cur ^ 1];
    uint32_t* R2 = rk[cur ^ 1];

    // 1. lowest rank in the unit
    uint32_t m = RANK_INF;
    for (uint32_t i = tid; i < n; i += NT) m = min(m, R[i]);
    m = wave_min_u32(m);
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
        const uint32_t i = r * 64 + lane;
        const uint64_t occ = __ballot(i < n && R[i] == m);
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
      const uint32_t i = r * 64 + lane;
      const uint64_t occ = __ballot(i < n && R[i] == m);
      const uint64_t s = leftmost_nonoverlapping(occ & ~(uint64_t)carry);
      if (lane == 0) sel[r] = s;
      const uint64_t valid = (n - r * 64 >= 64) ? ~0ull : ((1ull << (n - r * 64)) - 1ull);
      const uint64_t keep = valid & ~((s << 1) | (uint64_t)carry);
      keep_total += (uint32_t)__popcll(keep);
      carry = (uint32_t)(s >> 63);
    }
    if (tid == 0) sel[rows] = 0;  // sentinel row (only bit 0 is ever read)
    // 3. compaction
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
    }
    __syncthreads();
    uint32_t base = NW > 1 ? sm.wbase[wave] : 0u;
    const uint32_t n2 = NW > 1 ? sm.n_next : keep_total;
    uint32_t prevbit = (NW > 1 && r_lo > 0) ? (uint32_t)(sel[r_lo - 1] >> 63) : 0u;
    for (uint32_t r = r_lo; r < r_hi; ++r) {
      const uint32_t i = r * 64 + lane;
      const uint64_t s = sel[r];
      const uint64_t valid = (n - r * 64 >= 64) ? ~0ull : ((1ull << (n - r * 64)) - 1ull);
      const uint64_t keep = valid & ~((s << 1) | (uint64_t)prevbit);
      if ((keep >> lane) & 1ull) {
        const uint32_t k = base + bits_below(keep);
        const uint32_t my = (uint32_t)(s >> lane) & 1u;
        const uint32_t nx = lane < 63 ? (uint32_t)(s >> (lane + 1)) & 1u : (uint32_t)(sel[r + 1] & 1ull);
        I2[k] = my ? 256u + m : I[i];
        R2[k] = (my | nx) ? RANK_DIRTY : R[i];
      }
      base += (uint32_t)__popcll(keep);
      prevbit = (uint32_t)(s >> 63);
    }
    __syncthreads();
    n = n2;
    // 4. ranks of the pairs next to the merges
    for (uint32_t i = tid; i < n; i += NT) {
      if (R2[i] == RANK_DIRTY) R2[i] = i + 1 < n ? probe_rank(tb.slots, tb.nb, I2[i], I2[i + 1]) : RANK_INF;
    }
    __syncthreads();
    cur ^= 1;
  }
  const uint32_t* I = ids[cur];
  for (uint32_t i = tid; i < n; i += NT) out(i, I[i]);
  return n;
}

}  // namespace tt
