// The tile kernel: one block decides the pieces of 1,984 bytes of the request
// and encodes them, with no host round trip and no kernel boundary between
// pre-tokenization and BPE.
//
// Pre-tokenization.  The paper replaces the sequential leftmost-first regex
// scan by an equivalent per-character predicate: classify every character
// into letter / number / whitespace / other, form maximal same-class runs,
// and decide whether a character starts a piece from its offset in its run,
// at most four characters of lookback and a few per-run aggregates (Sec. 4.1,
// "Removing the sequential regex scan"; Sec. 4.2 lists the stages: decode,
// classify, runs, predicate, scans).  A block stages a 2,048-byte window (32
// bytes of context on each side of the bytes it owns) in LDS and every thread
// decodes and classifies two positions.  Runs that reach past the window are
// resolved without a second pass:
//   - backwards (cl100k: a number run's length mod 3, the class before a
//     CR/LF stretch) from run summaries that earlier blocks publish before
//     they wait on anything;
//   - forwards (cl100k: whether a whitespace stretch after CR/LF is the last
//     stretch of its run) by reading the bytes after the window, which only a
//     whitespace stretch longer than the window needs.
//
// Units.  For encoding, a piece is also cut at every byte position whose byte
// pair (b[q-1], b[q]) is the junction of no merge: the first merge that joins
// across a position has its left operand ending in b[q-1] and its right one
// starting with b[q], so no merge ever crosses such a position and the two
// sides are independent BPE problems.  The resulting units are numbered by a
// block scan.
//
// BPE (Sec. 4.2, "GPU BPE").  The block encodes every unit that starts in its
// bytes except its last one, whose end lies in a later tile: that unit is the
// "incoming" unit of the next tile that has a unit start, which learns its
// start from the position the earlier tiles publish right after their scan.
// Units go to the smallest execution unit that holds them (thread, wave, or
// the whole block over rows in LDS or, past the window size, global memory).
// Tokens are compacted in the tile and staged in global memory where the
// tile's bytes begin, so a tile's outputs never overlap another's; the emit
// kernel only has to place each tile's block of outputs.
//
// Block order is taken from an atomic ticket, so a block only ever waits on
// blocks that started before it, and every block publishes what later blocks
// wait for before it waits on anything itself.
#include "class_table.inc"
#include "class_table_o200k.inc"
#include "class_table_deepseek.inc"
#include "tt_bpe.h"
#include "tt_internal.h"
#include "tt_deepseek.h"
#include "tt_o200k.h"

namespace tt {

namespace {

// trailing-run summary of a tile (cl100k): bit 0 the run spans the whole tile,
// bits 1..2 its character count mod 3, bits 3..5 the class before it
constexpr uint32_t SUM_RUNALL = 1u;

// Words published for later blocks are self-contained values (the consumer
// reads nothing else the producer wrote), so relaxed device-scope atomics are
// enough: they are coherent across the chip without ordering other accesses.
__device__ __forceinline__ uint64_t ld_word(const uint64_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_word(uint64_t* p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// One lane waits for a word tagged with the call's epoch in its high half,
// sleeping between polls so that the wave does not flood the cache with loads.
__device__ __forceinline__ uint64_t wait_word(const uint64_t* p, uint32_t epoch) {
  uint64_t x = ld_word(p);
  while ((uint32_t)(x >> 32) != epoch) {
    __builtin_amdgcn_s_sleep(1);
    x = ld_word(p);
  }
  return x;
}

constexpr int CLS_L1_BYTES = 4352, CLS_L2_BYTES = TT_CLS_NBLOCKS * 64;

// The probed class table, staged in LDS by every block, and the code of every
// ASCII character (built by the block).
struct ClassLds {
  uint8_t l1[CLS_L1_BYTES] __attribute__((aligned(16)));
  uint8_t l2[CLS_L2_BYTES] __attribute__((aligned(16)));
  uint8_t asc[128];
};

// The 4-bit class table of a pattern whose pieces are walked (o200k-style,
// DeepSeek-style; same layout, room for the larger), staged in LDS by every
// block of that pattern, and the code of every ASCII character.
constexpr int WALK_NBLOCKS = TT_O2_NBLOCKS > TT_DS_NBLOCKS ? TT_O2_NBLOCKS : TT_DS_NBLOCKS;
struct O2Lds {
  uint8_t l1[4352] __attribute__((aligned(16)));
  uint8_t l2[WALK_NBLOCKS * 128] __attribute__((aligned(16)));
  uint8_t asc[128];
};

// 2-bit class of a non-ASCII code point from the probed table.
__device__ __forceinline__ uint32_t table_class(const ClassLds& ct, uint32_t cp) {
  const uint32_t blk = ct.l1[cp >> 8];
  const uint32_t b = ct.l2[blk * 64u + ((cp & 255u) >> 2)];
  return (b >> ((cp & 3u) * 2u)) & 3u;
}

__device__ __forceinline__ uint32_t letter_ident(uint32_t lower) {
  switch (lower) {
    case 's': return I_S;
    case 't': return I_T;
    case 'r': return I_R;
    case 'e': return I_E;
    case 'v': return I_V;
    case 'm': return I_M;
    case 'l': return I_L;
    case 'd': return I_D;
    default: return I_NONE;
  }
}

// Class and identity code of one code point.  Contraction letters are
// case-sensitive for GPT-2 and folded for cl100k, where the engine also folds
// U+017F (long s) to 's'.
// Code of one code point for the o200k-style pattern: its class only (the
// walks read apostrophes, "/" and contraction letters from the bytes).
__device__ __forceinline__ uint32_t o2_code(const O2Lds& t, uint32_t cp) {
  if (cp < 128u) {
    if ((cp - 'A') < 26u) return O2_UP;
    if ((cp - 'a') < 26u) return O2_LO;
    if ((cp - '0') < 10u) return O2_N;
    if (cp == 10u || cp == 13u) return O2_NL;
    if (cp == 32u || (cp - 9u) < 5u) return O2_WS;
    return O2_O;
  }
  return o2_table_class(t.l1, t.l2, cp);
}

// Code of one code point for the DeepSeek-style pattern: its class only.
// ASCII classes are computed: the ASCII table is built while the class table
// is still being staged.
__device__ __forceinline__ uint32_t ds_code(const O2Lds& t, uint32_t cp) {
  return cp < 128u ? ds_ascii_class(cp) : ds_table_class(t.l1, t.l2, cp);
}

// Code of a code point for a walked pattern.
template <int PAT>
__device__ __forceinline__ uint32_t walk_code(const O2Lds& t, uint32_t cp) {
  return PAT == TT_PATTERN_DEEPSEEK ? ds_code(t, cp) : o2_code(t, cp);
}

template <int PAT>
__device__ __forceinline__ uint32_t char_code(const ClassLds& ct, uint32_t cp) {
  uint32_t cls, id = I_NONE;
  if (cp < 128u) {
    if (((cp | 32u) - 'a') < 26u) cls = C_L;
    else if ((cp - '0') < 10u) cls = C_N;
    else if (cp == 10u || cp == 13u) cls = C_NL;
    else if (cp == 32u || (cp - 9u) < 5u) cls = C_WS;
    else cls = C_O;
    if (cp == 32u) id = I_SP;
    else if (cp == 39u) id = I_APO;
    else if (cls == C_L && (PAT == TT_PATTERN_CL100K || cp >= 'a')) id = letter_ident(cp | 32u);
  } else {
    uint32_t c2 = table_class(ct, cp);
    cls = c2 == 1u ? C_L : c2 == 2u ? C_N : c2 == 3u ? C_WS : C_O;
    if (PAT == TT_PATTERN_CL100K && cp == 0x17Fu) id = I_S;
  }
  return cls | (id << 3);
}

// Strict UTF-8 decode from bytes in registers, with selects only: the length
// of the sequence that starts with b0 (0 if it is invalid or longer than
// `avail`) and its code point.
__device__ __forceinline__ uint32_t decode_sel(uint32_t b0, uint32_t b1, uint32_t b2, uint32_t b3, uint32_t avail,
                                               uint32_t& cp) {
  const uint32_t len = b0 < 0x80u ? 1u : b0 < 0xC2u ? 0u : b0 < 0xE0u ? 2u : b0 < 0xF0u ? 3u : b0 < 0xF5u ? 4u : 0u;
  const uint32_t lo = b0 == 0xE0u ? 0xA0u : b0 == 0xF0u ? 0x90u : 0x80u;
  const uint32_t hi = b0 == 0xEDu ? 0x9Fu : b0 == 0xF4u ? 0x8Fu : 0xBFu;
  const bool ok1 = len < 2u || (b1 >= lo && b1 <= hi);
  const bool ok2 = len < 3u || (b2 & 0xC0u) == 0x80u;
  const bool ok3 = len < 4u || (b3 & 0xC0u) == 0x80u;
  const uint32_t c2 = ((b0 & 0x1Fu) << 6) | (b1 & 0x3Fu);
  const uint32_t c3 = ((b0 & 0x0Fu) << 12) | ((b1 & 0x3Fu) << 6) | (b2 & 0x3Fu);
  const uint32_t c4 = ((b0 & 0x07u) << 18) | ((b1 & 0x3Fu) << 12) | ((b2 & 0x3Fu) << 6) | (b3 & 0x3Fu);
  cp = len <= 1u ? b0 : len == 2u ? c2 : len == 3u ? c3 : c4;
  return (len != 0u && len <= avail && ok1 && ok2 && ok3) ? len : 0u;
}

// char_code for any code point of at most U+10FFFF, with selects only (both
// tables are read).
template <int PAT>
__device__ __forceinline__ uint32_t char_code_sel(const ClassLds& ct, uint32_t cp) {
  const uint32_t a = ct.asc[cp & 127u];
  const uint32_t c2 = table_class(ct, cp);
  const uint32_t cls = c2 == 1u ? C_L : c2 == 2u ? C_N : c2 == 3u ? C_WS : C_O;
  const uint32_t id = (PAT == TT_PATTERN_CL100K && cp == 0x17Fu) ? I_S : I_NONE;
  return cp < 128u ? a : (cls | (id << 3));
}

// Segmented char-count scan state for cl100k: has-head (bit 31), window index
// of the latest run head (bits 16..27), characters since that head (bits 0..15;
// or since the tile start when there is no head yet).
__device__ __forceinline__ uint32_t seg_combine(uint32_t a, uint32_t b) {
  return (b & 0x80000000u) ? b : ((a & 0xFFFF0000u) | ((a + b) & 0xFFFFu));
}
__device__ __forceinline__ bool seg_has(uint32_t s) { return (s & 0x80000000u) != 0; }
__device__ __forceinline__ int seg_head(uint32_t s) { return (int)((s >> 16) & 0x0FFFu); }
__device__ __forceinline__ uint32_t seg_cnt(uint32_t s) { return s & 0xFFFFu; }

template <typename F>
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v, int lane, F comb) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    uint32_t o = __shfl_up(v, d, 64);
    if (lane >= d) v = comb(o, v);
  }
  return v;
}


// The NW little-endian words of the L bytes at window index a (bytes past L
// read as zero), from aligned LDS words: NW + 1 word loads and one byte
// alignment per word.  Reads window bytes [a & ~3, a + 4 NW + 4).
template <int NW>
__device__ __forceinline__ void unit_words(const uint8_t* buf, uint32_t a, uint32_t L, uint32_t (&w)[NW]) {
  const uint32_t p = PT_PAD + a;
  const uint32_t* d = reinterpret_cast<const uint32_t*>(buf + (p & ~3u));
  const uint32_t sh = p & 3u;
  uint32_t x[NW + 1];
#pragma unroll
  for (int i = 0; i <= NW; ++i) x[i] = d[i];
#pragma unroll
  for (int i = 0; i < NW; ++i) {
    const uint32_t v = __builtin_amdgcn_alignbyte(x[i + 1], x[i], sh);
    const int rem = (int)L - 4 * i;  // bytes of word i inside the unit
    w[i] = rem >= 4 ? v : rem <= 0 ? 0u : (v & ((1u << (8 * rem)) - 1u));
  }
}

// ignore_merges: the internal ID of the vocabulary string equal to the L
// bytes byte(0 .. L) (2 <= L), or DICT_NONE.  Strings of up to DICT2_MAX bytes
// are probed with their bytes as the key (from the window when aw >= 0, i.e.
// the bytes start at window index aw); longer ones by two hashes of their
// bytes, confirmed by comparing the bytes with the stored string.
template <class ByteF>
__device__ uint32_t piece_find(const DevTables& tb, const uint8_t* buf, int64_t aw, uint32_t L, ByteF byte) {
  if (L <= (uint32_t)DICT2_MAX) {
    uint32_t kw[6] = {0u, 0u, 0u, 0u, 0u, 0u};
    if (aw >= 0 && aw + DICT2_MAX + 4 <= PT_WIN + 16) {
      unit_words(buf, (uint32_t)aw, L, kw);
    } else {
      for (uint32_t j = 0; j < L; ++j) kw[j >> 2] |= byte(j) << (8 * (j & 3));
    }
    if (L <= (uint32_t)DICT_MAX) return dict_find(tb.vdict, tb.vdnb, kw[0], kw[1], kw[2], L);
    return dict2_find(tb.vdict2, tb.vdnb2, kw, L);
  }
  uint32_t h1 = LONG_SEED1, h2 = LONG_SEED2;
  for (uint32_t j = 0; j < L; ++j) {
    const uint32_t b = byte(j);
    h1 = long_hash_step(h1, b);
    h2 = long_hash_step(h2, b);
  }
  h1 = long_hash_final(h1, L);
  h2 = long_hash_final(h2, L);
  const uint32_t b1 = 2u * bucket_of(h1, tb.vlnb), b2 = 2u * bucket_of(h2, tb.vlnb);
  const u32x4 e[4] = {tb.vlong[b1], tb.vlong[b1 + 1], tb.vlong[b2], tb.vlong[b2 + 1]};
  for (int i = 0; i < 4; ++i) {
    if (e[i].x != h1 || e[i].y != L) continue;
    bool same = true;
    for (uint32_t j = 0; j < L && same; ++j) same = tb.vblob[e[i].w + j] == byte(j);
    if (same) return e[i].z;
  }
  return DICT_NONE;
}

constexpr int MED_CAP = PT_WIN / (SMALL_MAX + 1) + 2;  // units of 17..WAVE_MAX bytes in a tile
// wave units are taken longest first, in classes of 8 bytes
constexpr int MED_CLASSES = (WAVE_MAX - SMALL_MAX + 7) / 8;
static_assert(SMALL_MAX < 64 && MED_CLASSES <= 64, "the start of each length (class) is one wave scan");
__device__ __forceinline__ uint32_t med_class(uint32_t L) { return (uint32_t)(WAVE_MAX - L) >> 3; }
constexpr int BIG_CAP = PT_WIN / (WAVE_MAX + 1) + 2;   // longer units in a tile
constexpr uint16_t U_INCOMING = 0xFFFFu;               // list entry for the incoming unit

// LDS of the classification phase and of the BPE phase share one region:
// nothing of the first is read after the unit scan, nothing of the second is
// written before it.
union PhaseMem {
  struct {
    union {
      ClassLds cls;           // character classes (GPT-2, cl100k)
      O2Lds o2;               // character classes (o200k, DeepSeek)
    };
    uint32_t join[2048];      // junction byte pairs of the merges
    uint8_t code[PT_PAD + PT_WIN + 16] __attribute__((aligned(16)));  // class/identity/doc-start codes
    union {
      int16_t run_end[PT_WIN];  // cl100k: window index of the head after a run's head
      struct {
        uint8_t o2piece[PT_WIN];  // walked patterns: 1 at the piece starts the walks find
        uint32_t o2bits[WALK_BITMAPS * WIN_WORDS];  // walked patterns: class-set bitmaps of the window
      };
    };
    uint32_t o2seg[PT_WIN / 32];    // walked patterns: segment starts (synchronizing positions, document starts)
    uint32_t nocut[PT_WIN / 32];    // ignore_merges: window positions no junction cut may split
  } a;
  struct {
    uint32_t tok[PT_WIN];     // tokens of unit k at tok[ustart[k] ..]
    uint16_t uoff[PT_WIN];    // first output of each unit within the tile
    uint16_t small[PT_OWN + 2];  // units of 3..16 bytes, sorted by length
    union {
      uint32_t wscr[PT_THREADS / 64][256];  // wave engine for 65..128 bytes: one area per wave
      struct {                              // block engine for 129..ROWS_LDS bytes
        uint32_t I0[ROWS_LDS], I1[ROWS_LDS], R0[ROWS_LDS], R1[ROWS_LDS];
        uint64_t sel[ROWS_LDS / 64 + 2];
      } rows;
    } x;
    uint32_t rk[SMALL_MAX - 1][TH_THREADS];  // thread engine: pair ranks, one column per thread
  } b;
};

struct PtShared {
  uint8_t buf[PT_PAD + PT_WIN + 16] __attribute__((aligned(16)));     // window bytes
  uint8_t dstart[PT_PAD + PT_WIN + 16] __attribute__((aligned(16)));  // 1 where a document starts
  PhaseMem ph;
  uint16_t ustart[PT_OWN + 2];  // window index of every unit start in the owned bytes
  uint16_t ucnt[PT_OWN + 2];    // tokens of each unit
  RowsShared<PT_THREADS / 64> rows;
  uint16_t med[MED_CAP];
  uint16_t big[BIG_CAP];
  uint32_t hist[SMALL_MAX + 1];  // small units per length, then where each length starts
  uint32_t hmed[MED_CLASSES];    // wave units per length class, then where each class starts
  uint32_t n_small, n_med, n_big;
  uint32_t med_next;             // next wave unit to take
  uint32_t wave_tot[PT_THREADS / 64];
  uint32_t tile;
  uint32_t inc_ids[SMALL_MAX];  // the incoming unit's tokens (thread engine)
  uint32_t s_prev;            // start of the incoming unit
  uint32_t prefix;            // outputs of all earlier tiles
  uint32_t err;               // invalid input in this tile or an earlier one
  uint32_t inc_cnt;           // its tokens
  uint32_t carry_n;           // cl100k: number-run chars before the tile, mod 3
  uint32_t carry_nlpre;       // cl100k: class before a CR/LF stretch entering the tile
  uint32_t cwave[PT_THREADS / 64];  // span export: per-wave sums
  int64_t o2_doc_after;          // walked patterns, batch: first document start after the window
  int64_t o2_last_s, o2_last_e;  // walked patterns: the tile's last piece (window indices)
  uint32_t o2_pub;               //   and whether it is published yet
  uint32_t whole[PT_WIN / 32];  // ignore_merges: starts of pieces that are vocabulary entries
  uint32_t cbase;             // span export: non-continuation bytes before the tile
  uint32_t ctile;             // span export: non-continuation bytes the tile owns
  int64_t doc_lo_idx;         // batch: first document start index touching the window
  int last_own;               // cl100k: window index of the tile's last own character
  // walked patterns: where the run of each run set through the window's end
  // ends past it, its last tracked character there, and whether wave 0 has
  // published them
  FarRuns far;
  // cl100k: a whitespace stretch after CR/LF that reaches the window's end
  int32_t ws_pend;            // its window index, or -1
  uint32_t ws_res;            // 1 when it is the last stretch of its run (read on past the window)
};

}  // namespace

// Word a tile publishes for the placement of its outputs:
//   bits 0..30 a count, bit 31 set when the count is inclusive (all outputs of
//   the tiles up to this one) rather than this tile's own, bit 32 set when
//   invalid input was seen (inclusive: in any tile up to this one), bits 33..63
//   the epoch of the call.
constexpr uint64_t PL_INC = 1ull << 31, PL_ERR = 1ull << 32;
constexpr int PL_EPOCH_SHIFT = 33;

// Decoupled look-back over the tiles' output counts (wave 0): publish this
// tile's count, then sum the counts of earlier tiles, newest first, until a
// tile whose published count is already inclusive.  A window of 64 earlier
// tiles is read at once and read again until every tile the sum needs has
// published (earlier tiles publish their own count before they look back, so
// the walk never waits on a tile that is itself waiting).  Returns the number
// of outputs before this tile, in every thread; the last tile also writes the
// output length, or the error.
//
// With span export (cagg != nullptr), wave 1 runs the same look-back over the
// tiles' non-continuation byte counts at the same time; each tile published
// its own count early, so this walk rarely waits.  The sum before the tile
// ends in sh.cbase.
__device__ __forceinline__ uint32_t lookback_counts(uint64_t* words, uint32_t t, uint64_t ep, uint32_t epoch,
                                                    int lane) {
  uint32_t prefix = 0;
  int64_t base = (int64_t)t - 1;
  for (;;) {
    const int64_t j = base - lane;
    uint64_t x = ep | PL_INC;  // before the first tile: an inclusive zero
    if (j >= 0) x = ld_word(&words[j]);
    const bool ready = (x >> PL_EPOCH_SHIFT) == (uint64_t)epoch;
    const uint64_t m_inc = __ballot(ready && (x & PL_INC));
    const uint64_t m_rdy = __ballot(ready);
    const int first = m_inc ? __ffsll((unsigned long long)m_inc) - 1 : 63;
    const uint64_t need = first >= 63 ? ~0ull : ((2ull << first) - 1ull);
    if ((m_rdy & need) != need) {
      __builtin_amdgcn_s_sleep(1);
      continue;
    }
    const uint32_t c = lane <= first ? (uint32_t)(x & 0x7FFFFFFFull) : 0u;
    prefix += (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_sum(c), 63);
    if (m_inc) break;
    base -= 64;
  }
  return prefix;
}

template <class Sh>
__device__ uint32_t place_tile(const Work& w, Sh& sh, uint32_t t, uint32_t count, bool bad, int tid, int lane,
                               int wave, uint64_t* cagg = nullptr, uint32_t c_tile = 0) {
  const uint64_t ep = (uint64_t)w.epoch << PL_EPOCH_SHIFT;
  if (cagg != nullptr) {
    if (t == 0) {
      if (tid == 0) {
        st_word(&cagg[0], ep | PL_INC | c_tile);
        sh.cbase = 0;
      }
    } else if (wave == 1) {
      const uint32_t cpre = lookback_counts(cagg, t, ep, w.epoch, lane);
      if (lane == 0) {
        st_word(&cagg[t], ep | PL_INC | (cpre + c_tile));
        sh.cbase = cpre;
      }
    }
  }
  uint64_t* pl = w.tile_agg;
  if (t == 0) {
    if (tid == 0) {
      st_word(&pl[0], ep | PL_INC | (bad ? PL_ERR : 0ull) | count);
      sh.prefix = 0;
      sh.err = bad ? 1u : 0u;
    }
  } else {
    if (tid == 0) st_word(&pl[t], ep | (bad ? PL_ERR : 0ull) | count);
    if (wave == 0) {
      uint32_t prefix = 0;
      bool err = bad;
      int64_t base = (int64_t)t - 1;
      for (;;) {
        const int64_t j = base - lane;
        uint64_t x = ep | PL_INC;  // before the first tile: an inclusive zero
        if (j >= 0) x = ld_word(&pl[j]);
        const bool ready = (x >> PL_EPOCH_SHIFT) == (uint64_t)w.epoch;
        const uint64_t m_inc = __ballot(ready && (x & PL_INC));
        const uint64_t m_rdy = __ballot(ready);
        const int first = m_inc ? __ffsll((unsigned long long)m_inc) - 1 : 63;
        const uint64_t need = first >= 63 ? ~0ull : ((2ull << first) - 1ull);
        if ((m_rdy & need) != need) {
          __builtin_amdgcn_s_sleep(1);
          continue;
        }
        const bool use = lane <= first;
        const uint32_t c = use ? (uint32_t)(x & 0x7FFFFFFFull) : 0u;
        prefix += (uint32_t)__builtin_amdgcn_readlane((int)wave_incl_sum(c), 63);
        err = err || __ballot(use && (x & PL_ERR)) != 0ull;
        if (m_inc) break;
        base -= 64;
      }
      if (lane == 0) {
        st_word(&pl[t], ep | PL_INC | (err ? PL_ERR : 0ull) | (prefix + count));
        sh.prefix = prefix;
        sh.err = err ? 1u : 0u;
      }
    }
  }
  __syncthreads();
  if (tid == 0) {
    if (w.doc_off != nullptr) w.tile_pre[t] = sh.prefix;
    if (t == w.n_tiles - 1) *w.out_len = sh.err ? (int64_t)TT_ERR_INVALID_UTF8 : (int64_t)(sh.prefix + count);
  }
  return sh.prefix;
}

// Phase stamps (a diagnostic build of the library, compiled with
// TT_PHASE_STAMPS; the product build has none of this): thread 0 of every tile
// writes the 100 MHz wall clock at each phase boundary into tt_phase_buf, slot
// k of the tile's TT_PHASE_SLOTS, and tt_phase_stamps copies them to the host.
// Slots: 0 entry, 1 ticket and tables, 2 window staged, 3 classified, 4 cl100k
// scan done, 5 predicate done, 6 dispatch done, 7 thread and wave engines
// done, 8 block engine done, 9 placement look-back done, 10 tokens written;
// inside the dispatch 11 unit scan done, 12 unit starts listed, 13 incoming
// unit found and dictionaries probed, 14 length lists built; inside the
// walked patterns' predicate 16 bitmaps built, 17 extra starts and the first
// wait done, 18 walks done, 19 flags done; 20 the incoming unit's start known
// (by the thread that dispatches it); 21 the predicate's per-position rules
// done (thread 0), 22 the cl100k read past the window and the vocabulary
// probes of ignore_merges done; 23 the block index; 24 + w: wave w done with
// the predicate (the same point as 5, per wave); 15 where the block runs (XCD
// in the high word, the hardware ID register in the low word).
#ifdef TT_PHASE_STAMPS
constexpr int TT_PHASE_SLOTS = 32, TT_PHASE_TILES = 8192;
__device__ unsigned long long tt_phase_buf[TT_PHASE_TILES * TT_PHASE_SLOTS];
#define TT_PHASE_BY(k, who)                                                                    \
  do {                                                                                         \
    if ((who) && t < (uint32_t)TT_PHASE_TILES) tt_phase_buf[(size_t)t * TT_PHASE_SLOTS + (k)] = wall_clock64(); \
  } while (0)
#else
#define TT_PHASE_BY(k, who) \
  do {                      \
  } while (0)
#endif
#define TT_PHASE(k) TT_PHASE_BY(k, tid == 0)

// MODE 0: split-level export; the outputs are the byte offsets of the pieces.
// MODE 1: encoding; the outputs are the (internal) IDs of the units' tokens.
// MODE 2: encoding with span export: also the byte start of every token and the
//         non-continuation byte count at every 4-byte word of the request.
template <int PAT, bool BATCH, int MODE, bool IGN>
__global__ __launch_bounds__(PT_THREADS) __attribute__((amdgpu_waves_per_eu(6))) void tile_kernel(Work w, DevTables tb) {
  constexpr bool SEG = MODE >= 1;
  constexpr bool SPANS = MODE == 2;
  __shared__ PtShared sh;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int64_t n = w.n;
#ifdef TT_PHASE_STAMPS
  const unsigned long long phase_s0 = wall_clock64();
#endif

  if (tid <= SMALL_MAX) sh.hist[tid] = 0;
  if (tid >= 64 && tid < 64 + MED_CLASSES) sh.hmed[tid - 64] = 0;
  if (IGN && tid < PT_WIN / 32) {
    sh.ph.a.nocut[tid] = 0;
    sh.whole[tid] = 0;
  }
  // the patterns whose pieces are walked between synchronizing positions
  constexpr bool DS = PAT == TT_PATTERN_DEEPSEEK;
  constexpr bool WALK = PAT == TT_PATTERN_O200K || DS;
  // the ticket's round trip (tickets are handed out one at a time) overlaps
  // the staging of the tables, which do not depend on the tile
  uint32_t ticket = 0;
  if (tid == 0) ticket = atomicAdd(&w.ctrl->tile_ticket, 1u);
  {
    // the class table (12.9 KB) is read once per block
    static_assert(CLS_L1_BYTES % 16 == 0 && CLS_L2_BYTES % 16 == 0, "class table staging uses 16-byte words");
    if (WALK) {
      constexpr int N1 = 4352 / 16, N2 = (DS ? TT_DS_NBLOCKS : TT_O2_NBLOCKS) * 128 / 16;
      const uint4* s1 = reinterpret_cast<const uint4*>(DS ? TT_DS_L1 : TT_O2_L1);
      const uint4* s2 = reinterpret_cast<const uint4*>(DS ? TT_DS_L2 : TT_O2_L2);
      uint4* d1 = reinterpret_cast<uint4*>(sh.ph.a.o2.l1);
      uint4* d2 = reinterpret_cast<uint4*>(sh.ph.a.o2.l2);
      for (int i = tid; i < N1 + N2; i += PT_THREADS) {
        if (i < N1) d1[i] = s1[i];
        else d2[i - N1] = s2[i - N1];
      }
      if (tid < 128) sh.ph.a.o2.asc[tid] = (uint8_t)walk_code<PAT>(sh.ph.a.o2, (uint32_t)tid);
    } else {
      constexpr int N1 = CLS_L1_BYTES / 16, N2 = CLS_L2_BYTES / 16;
      const uint4* s1 = reinterpret_cast<const uint4*>(TT_CLS_L1);
      const uint4* s2 = reinterpret_cast<const uint4*>(TT_CLS_L2);
      uint4* d1 = reinterpret_cast<uint4*>(sh.ph.a.cls.l1);
      uint4* d2 = reinterpret_cast<uint4*>(sh.ph.a.cls.l2);
      for (int i = tid; i < N1 + N2; i += PT_THREADS) {
        if (i < N1) d1[i] = s1[i];
        else d2[i - N1] = s2[i - N1];
      }
      if (tid < 128) sh.ph.a.cls.asc[tid] = (uint8_t)char_code<PAT>(sh.ph.a.cls, (uint32_t)tid);
    }
  }
  if (SEG) {
    // the junction bitmap (8 KB) is read once per block
    const uint4* src = reinterpret_cast<const uint4*>(tb.join);
    uint4* dst = reinterpret_cast<uint4*>(sh.ph.a.join);
    for (int i = tid; i < 512; i += PT_THREADS) dst[i] = src[i];
  }
  if (tid == 0) {
    sh.tile = ticket - w.ticket_base;
    sh.n_med = 0;
    sh.med_next = 0;
    sh.n_big = 0;
    sh.inc_cnt = 0;
    sh.ws_pend = -1;
  }
  if (tid < WALK_BITMAPS) sh.far.state[tid] = FAR_NONE;
  __syncthreads();
  const uint32_t t = wave_uniform(sh.tile);
  const uint32_t n_tiles = w.n_tiles;
  if (t >= n_tiles) return;
#ifdef TT_PHASE_STAMPS
  if (tid == 0 && t < (uint32_t)TT_PHASE_TILES) {
    tt_phase_buf[(size_t)t * TT_PHASE_SLOTS] = phase_s0;
    tt_phase_buf[(size_t)t * TT_PHASE_SLOTS + 20] = 0;  // (written later only by a tile with an incoming unit)
    tt_phase_buf[(size_t)t * TT_PHASE_SLOTS + 23] = blockIdx.x;
    // where the block runs: the XCD (XCC_ID register) and the hardware ID
    // register (compute unit, shader array and engine in bits 8-15)
    const uint32_t xcc = (uint32_t)__builtin_amdgcn_s_getreg((3 << 11) | 20) & 15u;
    const uint32_t hw = (uint32_t)__builtin_amdgcn_s_getreg((31 << 11) | 4);
    tt_phase_buf[(size_t)t * TT_PHASE_SLOTS + 15] = ((unsigned long long)xcc << 32) | hw;
  }
#endif
  TT_PHASE(1);
  const int64_t t0 = (int64_t)t * PT_OWN;
  const int64_t w0 = t0 - PT_HALO;

  auto inside = [&](int q) -> bool {
    int64_t p = w0 + q;
    return p >= 0 && p < n;
  };

  // ---- stage the window: 8 bytes per thread, one 64-bit load when possible --
  // LDS index of window position q is q + PT_PAD, for q in [-PT_PAD, PT_WIN + 16)
  auto stage_chunk = [&](int c) {  // window bytes [8c, 8c + 8)
    const int q0 = 8 * c;
    const int64_t p0 = w0 + q0;
    uint2 v = make_uint2(0u, 0u);
    if (p0 >= 0 && p0 + 8 <= n && ((reinterpret_cast<uintptr_t>(w.text + p0) & 7u) == 0)) {
      v = *reinterpret_cast<const uint2*>(w.text + p0);
    } else {
      uint32_t lo = 0, hi = 0;
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        int64_t p = p0 + k;
        uint32_t b = (p >= 0 && p < n) ? w.text[p] : 0u;
        if (k < 4) lo |= b << (8 * k);
        else hi |= b << (8 * (k - 4));
      }
      v = make_uint2(lo, hi);
    }
    *reinterpret_cast<uint2*>(&sh.buf[PT_PAD + q0]) = v;
    uint2 d = make_uint2(0u, 0u);
    if (p0 <= 0 && p0 + 8 > 0) d.x = (p0 == 0) ? 1u : 0u;  // the text start is a document start
    if (p0 < 0 && p0 + 8 > 0) {
      int k = (int)(-p0);
      if (k < 4) d.x = 1u << (8 * k);
      else d.y = 1u << (8 * (k - 4));
    }
    *reinterpret_cast<uint2*>(&sh.dstart[PT_PAD + q0]) = d;
  };
  {
    constexpr int NCH = PT_WIN / 8;  // chunks of the window proper
    if (tid < NCH) stage_chunk(tid);
    else if (tid < NCH + 3) stage_chunk(tid == NCH ? -1 : tid - 1);  // [-8, 0) and [PT_WIN, PT_WIN + 16)
  }
  if (BATCH) {
    if (tid == 0) {
      // first document start >= w0 - PT_PAD
      int lo = 0, hi = w.n_docs;  // search in doc_off[0..n_docs)
      while (lo < hi) {
        int mid = (lo + hi) >> 1;
        if (w.doc_off[mid] < w0 - PT_PAD) lo = mid + 1;
        else hi = mid;
      }
      sh.doc_lo_idx = lo;
      if (WALK) {
        int a = lo, b = w.n_docs;  // first document start >= w0 + PT_WIN
        while (a < b) {
          int mid = (a + b) >> 1;
          if (w.doc_off[mid] < w0 + PT_WIN) a = mid + 1;
          else b = mid;
        }
        sh.o2_doc_after = a < w.n_docs ? w.doc_off[a] : n;
      }
    }
  }
  __syncthreads();
  if (BATCH) {
    for (int64_t j = sh.doc_lo_idx + tid; j < w.n_docs; j += PT_THREADS) {
      int64_t d = w.doc_off[j];
      if (d >= w0 + PT_WIN + 16) break;
      if (d >= n) continue;
      sh.dstart[PT_PAD + (d - w0)] = 1;  // several empty documents may start here; all store the same value
    }
    __syncthreads();
  }

  TT_PHASE(2);
  // ---- decode, validate, classify ------------------------------------------
  // A thread's four positions are one aligned word of the window.  It reads
  // its word and the words on either side (bytes and document-start flags) and
  // decides everything from registers: a sequence starts at most three bytes
  // before a position it covers and ends at most three bytes after.  Four
  // ASCII bytes inside the text take their codes from the ASCII table.
  static_assert(PT_BPT == 4 && PT_PAD % 4 == 0, "classification works on aligned 4-byte words");
  bool bad = false;
  uint32_t nc_own = 0;  // span export: non-continuation bytes among the thread's own positions
  // (also counted again at the end, from the window bytes, instead of being kept)
  auto own_noncont = [&](uint32_t bytes, int q0, int64_t p0) -> uint32_t {
    const uint32_t cont = bytes & ~(bytes << 1) & 0x80808080u;  // bit 7 of each continuation byte
    uint32_t c = 0;
#pragma unroll
    for (int j = 0; j < PT_BPT; ++j) {
      const int q = q0 + j;
      const bool own = q >= PT_HALO && q < PT_HALO + PT_OWN && p0 + j >= 0 && p0 + j < n;
      c += (own && !((cont >> (8 * j + 7)) & 1u)) ? 1u : 0u;
    }
    return c;
  };
  {
    const int q0 = tid * PT_BPT;
    const uint32_t* bw = reinterpret_cast<const uint32_t*>(&sh.buf[PT_PAD + q0 - 4]);
    const uint32_t* dw = reinterpret_cast<const uint32_t*>(&sh.dstart[PT_PAD + q0 - 4]);
    const uint32_t bw0 = bw[0], bw1 = bw[1], bw2 = bw[2];
    const uint32_t dw0 = dw[0], dw1 = dw[1], dw2 = dw[2];
    const int64_t p0 = w0 + q0;  // text position of the first of the four
    if (SPANS) nc_own = own_noncont(bw1, q0, p0);
    uint32_t codes;
    if ((bw1 & 0x80808080u) == 0u && p0 >= 0 && p0 + PT_BPT <= n) {
      const uint8_t* asc = WALK ? sh.ph.a.o2.asc : sh.ph.a.cls.asc;
      codes = (uint32_t)asc[bw1 & 255u] | ((uint32_t)asc[(bw1 >> 8) & 255u] << 8) |
              ((uint32_t)asc[(bw1 >> 16) & 255u] << 16) | ((uint32_t)asc[bw1 >> 24] << 24);
      codes |= (dw1 & 0x01010101u) << 7;  // document starts (flags are 0 or 1)
    } else {
      const uint64_t blo = bw0 | ((uint64_t)bw1 << 32), bhi = bw1 | ((uint64_t)bw2 << 32);
      const uint64_t dlo = dw0 | ((uint64_t)dw1 << 32), dhi = dw1 | ((uint64_t)dw2 << 32);
      // r is relative to q0, in [-4, 8)
      auto byt = [&](int r) -> uint32_t {
        return r < 0 ? (uint32_t)(blo >> (8 * (r + 4))) & 255u : (uint32_t)(bhi >> (8 * r)) & 255u;
      };
      auto dst = [&](int r) -> bool {
        return ((r < 0 ? (uint32_t)(dlo >> (8 * (r + 4))) : (uint32_t)(dhi >> (8 * r))) & 255u) != 0u;
      };
      auto ins = [&](int r) -> bool { return p0 + r >= 0 && p0 + r < n; };
      codes = 0;
#pragma unroll
      for (int j = 0; j < PT_BPT; ++j) {
        const int q = q0 + j;
        const uint32_t b = byt(j);
        const bool in_j = ins(j);
        const bool own = q >= PT_HALO && q < PT_HALO + PT_OWN && in_j;
        const bool cont = (b & 0xC0u) == 0x80u;
        // a lead byte: its sequence, which a document start or the text end cuts
        uint32_t avail = 1;
        bool stop = false;
#pragma unroll
        for (int k = 1; k <= 3; ++k) {
          stop = stop || !ins(j + k) || dst(j + k);
          avail += stop ? 0u : 1u;
        }
        uint32_t cp = 0;
        const uint32_t len = decode_sel(b, byt(j + 1), byt(j + 2), byt(j + 3), avail, cp);
        // a continuation byte must lie inside the sequence of a lead byte at
        // most three bytes earlier, with no document start in between
        bool claimed = false, blocked = dst(j);
#pragma unroll
        for (int k = 1; k <= 3; ++k) {
          const uint32_t br = byt(j - k);
          const bool ok = ins(j - k), c = (br & 0xC0u) == 0x80u;
          const uint32_t ll = br < 0x80u ? 1u : br < 0xC2u ? 0u : br < 0xE0u ? 2u : br < 0xF0u ? 3u : br < 0xF5u ? 4u : 0u;
          claimed = claimed || (!blocked && ok && !c && ll > (uint32_t)k);
          blocked = blocked || !ok || !c || dst(j - k);
        }
        const uint32_t code = WALK ? ((!in_j || cont) ? O2_NONE : len == 0u ? O2_O : walk_code<PAT>(sh.ph.a.o2, cp))
                                 : (!in_j || cont) ? C_NONE : len == 0u ? C_O : char_code_sel<PAT>(sh.ph.a.cls, cp);
        bad = bad || (own && (cont ? !claimed : len == 0u));
        codes |= (code | (dst(j) ? CODE_DOCSTART : 0u)) << (8 * j);
      }
    }
    *reinterpret_cast<uint32_t*>(&sh.ph.a.code[PT_PAD + q0]) = codes;
    if (tid < 3) {  // positions outside [0, PT_WIN) carry no character for the rules
      const int qx = tid == 0 ? -8 : PT_WIN + 8 * (tid - 1);
      const uint32_t none4 = WALK ? 0x0F0F0F0Fu : 0x07070707u;
      *reinterpret_cast<uint2*>(&sh.ph.a.code[PT_PAD + qx]) = make_uint2(none4, none4);
    }
  }
  if (PAT == TT_PATTERN_CL100K)
    for (int q = tid; q < PT_WIN; q += PT_THREADS) sh.ph.a.run_end[q] = -1;
  if (WALK) *reinterpret_cast<uint32_t*>(&sh.ph.a.o2piece[tid * PT_BPT]) = 0u;
  if (SPANS) {
    const uint32_t nc_incl = wave_incl_sum(nc_own);
    if (lane == 63) sh.cwave[wave] = nc_incl;
  }
  const bool tile_bad = __syncthreads_or(bad) != 0;
  // span export: the tile's count is published before this block waits on
  // anything (the look-back that sums it runs at the end)
  if (SPANS && tid == 0) {
    uint32_t c_tile = 0;
    for (int v = 0; v < PT_THREADS / 64; ++v) c_tile += sh.cwave[v];
    sh.ctile = c_tile;
    st_word(&w.tile_cagg[t], ((uint64_t)w.epoch << PL_EPOCH_SHIFT) | c_tile);
  }

  TT_PHASE(3);
  // ---- neighbour helpers (window indices; -1 = none) ----------------------
  auto code_at = [&](int q) -> uint32_t { return sh.ph.a.code[PT_PAD + q]; };
  auto cls = [&](int q) -> uint32_t { return code_cls(code_at(q)); };
  auto ident = [&](int q) -> uint32_t { return code_id(code_at(q)); };
  auto prev = [&](int q) -> int {
    if (code_at(q) & CODE_DOCSTART) return -1;
    for (int r = q - 1; r >= 0; --r) {
      if (!inside(r)) return -1;
      if (code_cls(code_at(r)) != C_NONE) return r;
    }
    return -1;
  };
  auto next = [&](int q) -> int {
    for (int r = q + 1; r < PT_WIN + 8; ++r) {
      if (!inside(r)) return -1;
      const uint32_t c = code_at(r);
      if (c & CODE_DOCSTART) return -1;
      if (code_cls(c) != C_NONE) return r;
    }
    return -1;
  };
  auto is_char = [&](int q) -> bool { return inside(q) && code_cls(code_at(q)) != C_NONE; };
  auto is_w = [](uint32_t c) -> bool { return c == C_WS || c == C_NL; };

  // Suffix of a contraction starting at letter q: 1 or 2 letters, or 0.
  auto suffix_len = [&](int q) -> int {
    uint32_t a = ident(q);
    if (a == I_S || a == I_T || a == I_M || a == I_D) return 1;
    if (a == I_R || a == I_V || a == I_L) {
      int q1 = next(q);
      if (q1 >= 0) {
        uint32_t b = ident(q1);
        if ((a == I_R && b == I_E) || (a == I_V && b == I_E) || (a == I_L && b == I_L)) return 2;
      }
    }
    return 0;
  };
  // Letter q starts a contraction suffix: the apostrophe before it begins a
  // match, i.e. it is a one-character "other" run not preceded by U+0020.
  auto contraction_len_at = [&](int q) -> int {
    int p1 = prev(q);
    if (p1 < 0 || ident(p1) != I_APO) return 0;
    int p2 = prev(p1);
    if (p2 >= 0 && (cls(p2) == C_O || ident(p2) == I_SP)) return 0;
    return suffix_len(q);
  };
  // Letter q (inside a letter run) is the first letter after a contraction.
  auto contraction_ends_here = [&](int q) -> bool {
    int p1 = prev(q);
    if (contraction_len_at(p1) == 1) return true;
    int p2 = prev(p1);
    return p2 >= 0 && cls(p2) == C_L && contraction_len_at(p2) == 2;
  };

  // ---- the codes around the thread's positions, in registers ---------------
  // cr(r) is the code of window position qb + r for r in [-8, 8): enough to
  // find the characters on either side of the thread's positions (and the one
  // before that), which are at most four bytes away in valid text.
  const int qb = tid * PT_BPT;
  const uint32_t* cwp = reinterpret_cast<const uint32_t*>(&sh.ph.a.code[PT_PAD + qb - 8]);
  const uint32_t cw0 = cwp[0], cw1 = cwp[1], cw2 = cwp[2], cw3 = cwp[3];
  auto cr = [&](int r) -> uint32_t {
    const int i = r + 8;
    const uint32_t lo = (i & 4) ? cw1 : cw0, hi = (i & 4) ? cw3 : cw2;
    return (((i & 8) ? hi : lo) >> ((i & 3) * 8)) & 255u;
  };
  // an apostrophe one byte before position qb + r (a contraction can start at
  // qb + r only then), or two or three bytes before (a contraction can end just
  // before qb + r only then: the suffix is one or two ASCII letters, or U+017F)
  auto apo_at = [&](int r) -> bool { return code_id(cr(r)) == I_APO; };
  // The character before window position qb + r (r in [-4, 8)) and its code,
  // from the register window: in valid text it starts at most four bytes
  // before (in invalid text, whose output is discarded, the search stops
  // there).  Returns its distance, 0 when there is none.
  auto prev_reg = [&](int r, uint32_t& pc) -> uint32_t {
    uint32_t d = 0, x = 0;
#pragma unroll
    for (int k = 4; k >= 1; --k) {
      const uint32_t c = cr(r - k);
      const bool ch = code_cls(c) != C_NONE;
      d = ch ? (uint32_t)k : d;
      x = ch ? c : x;
    }
    pc = x;
    return (cr(r) & CODE_DOCSTART) ? 0u : d;
  };
  // Whether a character follows position qb + r (r in [-8, 4)) in the same
  // document, within four bytes, and its code.
  auto next_reg = [&](int r, uint32_t& nc) -> bool {
    bool found = false, stop = false;
    uint32_t x = 0;
#pragma unroll
    for (int k = 1; k <= 4; ++k) {
      const uint32_t c = cr(r + k);
      const bool ds = (c & CODE_DOCSTART) != 0u, ch = code_cls(c) != C_NONE;
      found = found || (!stop && !ds && ch);
      x = (!stop && !ds && ch) ? c : x;
      stop = stop || ds || ch;
    }
    nc = x;
    return found;
  };

  // ---- cl100k: run scan, run ends, summaries, carries ----------------------
  // scan element of window position qb + j: a run head restarts the char count
  auto elem_of = [&](int j) -> uint32_t {
    const int q = qb + j;
    const uint32_t c = cr(j);
    if (q < PT_HALO || code_cls(c) == C_NONE) return 0u;
    uint32_t pc = 0;
    const bool head = prev_reg(j, pc) == 0u || code_cls(pc) != code_cls(c);
    return head ? (0x80000000u | ((uint32_t)q << 16) | 1u) : 1u;
  };
  uint32_t elems[PT_BPT];
#pragma unroll
  for (int j = 0; j < PT_BPT; ++j) elems[j] = PAT == TT_PATTERN_CL100K ? elem_of(j) : 0u;
  uint32_t s0 = 0;  // scan state before the thread's first position
  if (PAT == TT_PATTERN_CL100K) {
    // elements over window indices [HALO, WIN)
    uint32_t agg = 0;
#pragma unroll
    for (int j = 0; j < PT_BPT; ++j) agg = seg_combine(agg, elems[j]);
    uint32_t inc = wave_incl_scan(agg, lane, seg_combine);
    if (lane == 63) sh.wave_tot[wave] = inc;
    uint32_t lex = __shfl_up(inc, 1, 64);
    if (lane == 0) lex = 0;
    __syncthreads();
    uint32_t wpre = 0;
    for (int v = 0; v < wave; ++v) wpre = seg_combine(wpre, sh.wave_tot[v]);
    s0 = seg_combine(wpre, lex);
    // each run head records itself as the end of the previous run
    const int own_end = (int)(n - w0 < PT_HALO + PT_OWN ? n - w0 : PT_HALO + PT_OWN);
    int last_q = -1;
    uint32_t last_st = 0;
    {
      uint32_t st = s0;
#pragma unroll
      for (int j = 0; j < PT_BPT; ++j) {
        const int q = qb + j;
        const uint32_t e = elems[j];
        if ((e & 0x80000000u) && seg_has(st)) sh.ph.a.run_end[seg_head(st)] = (int16_t)q;
        st = seg_combine(st, e);
        if (q >= PT_HALO && q < own_end && e != 0u) {
          last_q = q;
          last_st = st;
        }
      }
    }
    // summary of the tile's trailing run (own range), published before waiting
    // on any other block; the thread holding the last own character publishes
    if (tid == 0) sh.last_own = -1;
    __syncthreads();
    if (last_q >= 0) atomicMax(&sh.last_own, last_q);
    __syncthreads();
    const int s_last = sh.last_own;
    if (s_last < 0) {
      if (tid == 0) st_word(&w.tile_sum[t], ((uint64_t)w.epoch << 32) | SUM_RUNALL);
    } else if (s_last == last_q) {
      uint32_t sum = (seg_cnt(last_st) % 3u) << 1;
      if (seg_has(last_st)) {
        int hp = prev(seg_head(last_st));
        sum |= (hp >= 0 ? cls(hp) : (uint32_t)C_NONE) << 3;
      } else {
        sum |= SUM_RUNALL;
      }
      st_word(&w.tile_sum[t], ((uint64_t)w.epoch << 32) | sum);
    }
    // carries for a run entering the tile from the left
    if (tid == 0) {
      sh.carry_n = 0;
      sh.carry_nlpre = C_NONE;
    }
    __syncthreads();
    if (wave == 0) {
      int f = -1;  // first own character
      for (int q = PT_HALO; q < PT_HALO + PT_OWN; ++q)
        if (is_char(q)) {
          f = q;
          break;
        }
      // a number run continuing into the tile needs its length so far; a
      // CR/LF stretch ending at or after the tile start needs the class
      // before it (the first own character may be the whitespace after it)
      bool need = false;
      if (f >= 0 && t > 0) {
        int p = prev(f);
        need = p >= 0 && ((cls(p) == C_N && cls(f) == C_N) || cls(p) == C_NL);
      }
      // walk back tile by tile (usually one step) until a tile whose trailing
      // run does not span it
      if (need && lane == 0) {
        uint32_t acc = 0, pre = C_NONE;
        for (int64_t j = (int64_t)t - 1; j >= 0; --j) {
          const uint64_t x = wait_word(&w.tile_sum[j], w.epoch);
          const uint32_t v = (uint32_t)x;
          acc += (v >> 1) & 3u;
          if (!(v & SUM_RUNALL)) {
            pre = (v >> 3) & 7u;
            break;
          }
        }
        sh.carry_n = acc % 3u;
        sh.carry_nlpre = pre;
      }
    }
    __syncthreads();
  }

  // rule 2 of cl100k: is the whitespace stretch starting at q (after CR/LF)
  // the last stretch of its whitespace run?  1 yes, 0 no, -1 when the stretch
  // reaches the window's end and the answer lies in the text after it (the
  // block reads on there together, below)
  auto ws_stretch_is_last = [&](int q) -> int {
    int e = sh.ph.a.run_end[q];
    if (e >= 0) return ((code_at(e) & CODE_DOCSTART) || cls(e) != C_NL) ? 1 : 0;
    if (w0 + PT_WIN >= n) return 1;  // the run reaches the end of the text
    return -1;
  };

  TT_PHASE(4);
  // ---- piece-start predicate ----------------------------------------------
  // The run-local rules, from the codes of the position, of the characters
  // before and after it (register window) and, for cl100k, the run scan.  The
  // cheap cases are selects; contractions (an apostrophe one to three bytes
  // back), whitespace after CR/LF and a letter after a lone symbol branch.
  uint32_t flags = 0;
  if (WALK) {
    // o200k- and DeepSeek-style: segment starts are document starts,
    // synchronizing positions (their two neighbouring characters form a
    // transition of o2_sync or ds_sync) and two whitespace cases that start a
    // piece for every left context given the text to their right (below);
    // the pieces of a segment come from running the pattern's alternatives
    // from its start, one lane per segment
    auto walk_ws = [&](uint32_t cl) -> bool { return DS ? (cl == DS_SP || cl == DS_WS) : cl == O2_WS; };
    auto walk_solid = [&](uint32_t cl) -> bool {  // not whitespace (DeepSeek-style: and of the rest group)
      return DS ? (cl != DS_SP && cl != DS_WS && cl != DS_NL && ds_group(cl) == 0u)
                : (cl != O2_WS && cl != O2_NL && cl != O2_NONE);
    };
    // Everything here is selects over the register window and table bits
    // (o2_sync_bits, ds_sync_bits, the bitmap class masks): a switch over
    // classes would be a tree of divergent branches.
    // the window bytes qb - 4 .. qb + 3: the character before a position
    // starts at most four bytes back
    const uint32_t bwlo = *reinterpret_cast<const uint32_t*>(&sh.buf[PT_PAD + qb - 4]);
    const uint32_t bwhi = *reinterpret_cast<const uint32_t*>(&sh.buf[PT_PAD + qb]);
    auto wbyte = [&](int r) -> uint32_t {  // r in [-4, 4)
      return ((r < 0 ? bwlo : bwhi) >> (8 * (r & 3))) & 255u;
    };
    uint32_t seg = 0;
    uint32_t nib[WALK_BITMAPS];  // the class-set bitmaps' bits of the thread's four positions
#pragma unroll
    for (int k = 0; k < WALK_BITMAPS; ++k) nib[k] = 0;
#pragma unroll
    for (int j = 0; j < PT_BPT; ++j) {
      const int q = qb + j;
      const uint32_t c = cr(j);
      const uint32_t cl = c & 15u;
      const bool in_q = inside(q);
      const bool dstart = (c & CODE_DOCSTART) != 0u;
      // the character before q: its distance, class and (one-byte) byte
      int k = 0;
      uint32_t xc = O2_NONE, xb = 0x80u;
#pragma unroll
      for (int d = 4; d >= 1; --d) {
        const bool lead = (cr(j - d) & 15u) != O2_NONE;
        k = lead ? d : k;
        xc = lead ? (cr(j - d) & 15u) : xc;
        xb = lead ? (d == 1 ? wbyte(j - 1) : 0x80u) : xb;
      }
      const bool pair = (k > 0) & (q - k >= 0) &
                        (DS ? ds_sync_bits(xc, cl) : o2_sync_bits(xc, cl, xb, wbyte(j)));
      // one-byte whitespace before a character that is not whitespace, in
      // the same document (and, DeepSeek-style, the same group stretch): no
      // piece holds whitespace past its first character unless the piece
      // ends with whitespace or CR/LF (the alternatives that take whitespace
      // runs), and those cannot end before a character that is not
      // whitespace inside the stretch, so a piece starts here whatever the
      // left context
      const uint32_t c2 = cr(j + 1);
      const bool ws_solid = walk_ws(cl) & inside(q + 1) & ((c2 & CODE_DOCSTART) == 0u) & walk_solid(c2 & 15u);
      seg |= (uint32_t)(in_q & (cl != O2_NONE) & (dstart | pair | ws_solid)) << j;
      // the class-set bitmaps (tt_o200k.h): the sets of a character at its
      // first byte, the run sets at its continuation bytes, nothing at
      // document starts and outside the text; and the ASCII digits
      const bool in_b = in_q & !dstart;
#pragma unroll
      for (int kb = 0; kb < WALK_BITMAPS; ++kb) {
        const uint32_t cls_k = DS ? ds_bitmap_classes(kb) : o2_bitmap_classes(kb);
        const bool bit = kb == WB_DIGITS ? wbyte(j) - (uint32_t)'0' < 10u : ((cls_k >> cl) & 1u) != 0u;
        nib[kb] |= (uint32_t)(in_b & bit) << j;
      }
    }
    // A bitmap word holds the four positions of eight consecutive lanes: the
    // last lane of the eight stores the word, ORed together over DPP row
    // shifts (no atomics, and no clearing beforehand).
    static_assert(PT_BPT == 4 && PT_THREADS * PT_BPT == PT_WIN, "eight lanes per bitmap word");
    auto store_word = [&](uint32_t* words, uint32_t nib4) {
      int x = (int)(nib4 << (qb & 31));
      x |= __builtin_amdgcn_update_dpp(0, x, 0x111, 0xF, 0xF, true);  // row_shr:1
      x |= __builtin_amdgcn_update_dpp(0, x, 0x112, 0xF, 0xF, true);  // row_shr:2
      x |= __builtin_amdgcn_update_dpp(0, x, 0x114, 0xF, 0xF, true);  // row_shr:4
      if ((lane & 7) == 7) words[qb >> 5] = (uint32_t)x;
    };
    store_word(sh.ph.a.o2seg, seg);
#pragma unroll
    for (int kb = 0; kb < WALK_BITMAPS; ++kb) store_word(&sh.ph.a.o2bits[kb * WIN_WORDS], nib[kb]);
    if (tid == 0) {  // the tile's last piece, until a walk finds it (kept only for invalid text)
      sh.o2_last_s = PT_HALO;
      sh.o2_last_e = n - w0 < PT_HALO + PT_OWN ? n - w0 : PT_HALO + PT_OWN;
      sh.o2_pub = 0;
    }
    __syncthreads();
    TT_PHASE(16);
    const O2View v{(lds_u8*)sh.buf, (lds_u8*)sh.ph.a.code, (lds_u8*)sh.ph.a.o2.l1, (lds_u8*)sh.ph.a.o2.l2,
                   w.text, w0, n, BATCH ? sh.o2_doc_after : n, (lds_u32*)sh.ph.a.o2bits,
                   (lds_u8*)sh.ph.a.o2.asc, (lds_far*)&sh.far};
    const int64_t own_end = n - w0 < PT_HALO + PT_OWN ? n - w0 : PT_HALO + PT_OWN;
    auto segbit = [&](int64_t q) -> bool { return q >= 0 && q < PT_WIN && ((sh.ph.a.o2seg[q >> 5] >> (q & 31)) & 1u); };
    {
      // Whitespace right after CR/LF whose whitespace run holds no further
      // CR/LF starts a piece whatever the left context: the CR/LF ends a
      // symbol piece's CR/LF tail or a piece of the CR/LF alternative, which
      // runs to the last CR/LF of its whitespace run.  The run is read from
      // the bitmaps, so these marks come after the barrier; a walk of another
      // wave that does not see one yet walks on through it, to the same
      // pieces.
      uint32_t add = 0;
#pragma unroll
      for (int j = 0; j < PT_BPT; ++j) {
        const int q = qb + j;
        const uint32_t c = cr(j);
        if (((seg >> j) & 1u) || q < 1 || !inside(q) || !inside(q - 1) || (c & CODE_DOCSTART) || !walk_ws(c & 15u) ||
            (cr(j - 1) & 15u) != (DS ? (uint32_t)DS_NL : (uint32_t)O2_NL))
          continue;
        const int64_t r = win_next_zero(v.bits + (DS ? DSB_SP : O2B_SP) * WIN_WORDS, q);
        if (r < PT_WIN && win_last_one(v.bits + (DS ? DSB_NL : O2B_NL) * WIN_WORDS, q, r) < 0) add |= 1u << j;
      }
      if (add) {
        seg |= add;
        atomicOr(&sh.ph.a.o2seg[qb >> 5], add << (qb & 31));
      }
    }
    // one loop per lane, one piece per step: the lane's walk starts in order
    // (thread 0's continued segment first, then its own segment starts), so
    // a wave runs as long as its busiest lane, not its longest segment of
    // every start
    // thread 0 first walks the segment that the tile's first bytes continue,
    // from its start in the left context, else from the end of the last piece
    // of the previous tile (which holds the previous tile's last byte, so its
    // end is at or after this tile's first byte).  When that piece also holds
    // this tile's last byte, the tile has no piece start of its own and
    // passes the piece on without walking: a long piece is walked once, by the
    // tile it starts in, not again by every tile it covers.
    // The last piece of the tile (the one that holds its last byte) is kept in
    // last_s / last_e (their defaults were set before the barrier above, so
    // that no walk's write can come before them), and the next tile continues
    // from it: the lane that finds it publishes it at once (the next tile may
    // be waiting for it), not after the tile's other walks.
    auto publish_last = [&](int64_t ps, int64_t pe) {
      const uint64_t ep = (uint64_t)w.epoch << 32;
      st_word(&w.tile_end[t], ep | (uint32_t)(w0 + pe));
      st_word(&w.tile_sum[t], ep | (uint32_t)(w0 + ps));
      sh.o2_pub = 1u;
    };
    int64_t first = -1;
    if (tid == 0 && !segbit(PT_HALO)) {
      for (int q = PT_HALO - 1; q >= 0 && first < 0; --q)
        if (segbit(q)) first = q;
      if (first < 0 && t == 0) first = PT_HALO;  // (invalid text: no character at the text start)
      if (first < 0) {
        const uint64_t xs = wait_word(&w.tile_sum[t - 1], w.epoch);
        const uint64_t xe = wait_word(&w.tile_end[t - 1], w.epoch);
        const int64_t ps = (int64_t)(uint32_t)xs - w0, pe = (int64_t)(uint32_t)xe - w0;
        if (pe >= own_end) {
          sh.o2_last_s = ps;
          sh.o2_last_e = pe;
          publish_last(ps, pe);
        } else {
          first = pe < PT_HALO ? PT_HALO : pe;  // (pe < PT_HALO only for invalid text)
        }
      }
    }
    TT_PHASE(17);
    uint32_t todo = 0;  // bit j: own position qb + j starts a segment to walk
#pragma unroll
    for (int j = 0; j < PT_BPT; ++j)
      if (((seg >> j) & 1u) && qb + j >= PT_HALO && qb + j < own_end) todo |= 1u << j;
    // The wave's segment starts are dealt to its lanes in turn (a lane whose
    // four bytes hold several starts does not walk them all): rank r counts
    // the starts at byte j = 0 of every lane first, then j = 1, and so on;
    // lane l walks ranks l, l + 64, ...
    const uint64_t sb0 = __ballot(todo & 1u), sb1 = __ballot(todo & 2u), sb2 = __ballot(todo & 4u),
                   sb3 = __ballot(todo & 8u);
    const uint32_t sn0 = (uint32_t)__builtin_popcountll(sb0), sn1 = (uint32_t)__builtin_popcountll(sb1),
                   sn2 = (uint32_t)__builtin_popcountll(sb2);
    const uint32_t n_seg = sn0 + sn1 + sn2 + (uint32_t)__builtin_popcountll(sb3);
    auto seg_at = [&](uint32_t r) -> int64_t {  // window index of the start of rank r (< n_seg)
      uint64_t m = sb0;
      int j = 0;
      if (r >= sn0) { r -= sn0; m = sb1; j = 1; }
      if (j == 1 && r >= sn1) { r -= sn1; m = sb2; j = 2; }
      if (j == 2 && r >= sn2) { r -= sn2; m = sb3; j = 3; }
      return (int64_t)((wave * 64 + (int)select_bit64(m, r)) * PT_BPT + j);
    };
    uint32_t rank = lane;
    int64_t s = first;
    bool on_first = first != -1;
    if (!on_first && rank < n_seg) {
      s = seg_at(rank);
      rank += 64;
    }
    bool active = on_first || s != -1;
    // A walk whose piece needs a run through the window's end (rare) stops
    // at that piece; when every lane of the wave has stopped or finished,
    // the wave finds the runs asked for and those walks go on.
    int need = -1;
#pragma unroll 1
    for (;;) {
#pragma unroll 1
      while (active) {
        if (s >= PT_HALO) sh.ph.a.o2piece[s] = 1;  // (s < own_end <= PT_WIN)
        // A run of numbers is cut in threes from its head whatever surrounds it
        // (no other alternative takes a number), so from a piece start inside a
        // run of ASCII digits every third byte starts a piece: the full chunks
        // that end by own_end are marked in one step (a run of thousands of
        // digits is one short loop, not a piece per step).
        int64_t full = 0;  // full chunks of three ASCII digits from s
        if ((uint32_t)sh.buf[PT_PAD + s] - (uint32_t)'0' < 10u) {
          const int64_t dig = win_next_zero(v.bits + WB_DIGITS * WIN_WORDS, s) - s;
          full = (dig < own_end - s ? dig : own_end - s) / 3;
        }
        int64_t ps = s, e;
        if (full >= 1) {
#pragma unroll 1
          for (int64_t k = 1; k < full; ++k)
            if (s + 3 * k >= PT_HALO) sh.ph.a.o2piece[s + 3 * k] = 1;
          ps = s + 3 * (full - 1);
          e = s + 3 * full;
        } else {
          e = DS ? ds_piece_end(v, s) : o2_piece_end(v, s);
          if (e < 0) {  // the piece needs the run through the window's end of bitmap -1 - e
            need = (int)(-1 - e);
            break;
          }
        }
        if (e >= own_end) {  // the tile's last piece (one lane finds it)
          sh.o2_last_s = ps;
          sh.o2_last_e = e;
          publish_last(ps, e);
        }
        if (e < own_end && !segbit(e)) {
          s = e;
        } else if (rank < n_seg) {
          on_first = false;
          s = seg_at(rank);
          rank += 64;
        } else {
          active = false;
        }
      }
      uint32_t sets = need >= 0 ? 1u << need : 0u;  // the bitmaps the wave's walks ask for
#pragma unroll
      for (int d = 1; d < 64; d <<= 1) sets |= (uint32_t)__shfl_xor((int)sets, d, 64);
      if (sets == 0u) break;
      if (DS) ds_far_serve(v, sets);
      else o2_far_serve(v, sets);
      need = -1;
    }
    __syncthreads();
    TT_PHASE(18);
    const uint32_t pw = *reinterpret_cast<const uint32_t*>(&sh.ph.a.o2piece[qb]);
    flags = (pw & 1u) | ((pw >> 7) & 2u) | ((pw >> 14) & 4u) | ((pw >> 21) & 8u);
    // (no walk found the last piece only in invalid text)
    if (tid == 0 && sh.o2_pub == 0u) publish_last(sh.o2_last_s, sh.o2_last_e);
  }
  if (WALK) TT_PHASE(19);
  uint32_t scan_st = s0;  // cl100k: scan state before position q
#pragma unroll
  for (int j = 0; j < (WALK ? 0 : PT_BPT); ++j) {
    const int q = qb + j;
    const uint32_t ex = scan_st;
    if (PAT == TT_PATTERN_CL100K) scan_st = seg_combine(scan_st, elems[j]);
    const uint32_t cq = cr(j);
    const uint32_t c0 = code_cls(cq);
    if (q < PT_HALO || q >= PT_HALO + PT_OWN || c0 == C_NONE) continue;
    uint32_t cp1 = 0, cn1 = 0;
    const uint32_t d1 = prev_reg(j, cp1);
    const bool hn = next_reg(j, cn1);
    const uint32_t c1 = code_cls(cp1);
    const bool w0c = is_w(c0), w1c = is_w(c1);
    const bool sp1 = code_id(cp1) == I_SP;
    const bool run_last = hn && !is_w(code_cls(cn1));  // a following character that is not whitespace
    const bool apo1 = apo_at(j - 1), apo23 = apo_at(j - 2) || apo_at(j - 3);
    bool start;
    if (PAT == TT_PATTERN_GPT2) {
      start = w0c ? (!w1c || run_last) : (c1 != c0 && !sp1);
      if (!w0c && c0 == C_L && (apo1 || apo23)) {
        if (c1 == c0) start = apo23 && contraction_ends_here(q);
        else if (!sp1 && apo1 && contraction_len_at(q) > 0) start = false;
      }
    } else {
      if (w0c) {
        start = !w1c ? !(c1 == C_O && c0 == C_NL) : (c0 == C_NL ? false : run_last);
        if (w1c && c0 != C_NL && c1 == C_NL) {
          // first whitespace after a CR/LF stretch
          uint32_t pre;
          if (seg_has(ex)) {
            int hp = prev(seg_head(ex));
            pre = hp >= 0 ? cls(hp) : (uint32_t)C_NONE;
          } else {
            pre = sh.carry_nlpre;
          }
          if (pre == C_O) {
            start = true;
          } else {
            const int r = ws_stretch_is_last(q);
            start = r > 0;
            if (r < 0) sh.ws_pend = q;  // (one stretch at most reaches the window's end)
          }
        }
      } else if (c0 == C_N) {
        const uint32_t off = seg_cnt(ex) + (seg_has(ex) ? 0u : sh.carry_n);
        start = c1 != C_N || off % 3u == 0u;
      } else if (c0 == C_O) {
        start = c1 != C_O && !sp1;
      } else {  // letter
        start = c1 != C_L && c1 != C_WS;
        if (c1 == C_O) {
          // a lone symbol not preceded by U+0020 is the letter run's prefix
          uint32_t cp2 = 0;
          const uint32_t d2 = d1 == 1u ? prev_reg(j - 1, cp2) : d1 == 2u ? prev_reg(j - 2, cp2)
                            : d1 == 3u ? prev_reg(j - 3, cp2) : prev_reg(j - 4, cp2);
          start = d2 != 0u && (code_cls(cp2) == C_O || code_id(cp2) == I_SP);
        }
        if (apo1 || apo23) {
          if (c1 == C_L) start = apo23 && contraction_ends_here(q);
          else if (apo1 && contraction_len_at(q) > 0) start = false;
        }
      }
    }
    if (d1 == 0u) start = true;
    if (start) flags |= 1u << j;
  }
  TT_PHASE(21);
  if (PAT == TT_PATTERN_CL100K) {
    // the whitespace stretch after CR/LF that reaches the window's end, if
    // any: the block reads on past the window
    __syncthreads();
    const int pend = sh.ws_pend;
    if (pend >= 0) {
      // Wave 0 reads on, 16 bytes per lane per step, to the first byte that is
      // not plain ASCII whitespace (space, tab, VT, FF) and decodes the
      // character there (CR/LF: not the run's last stretch; other whitespace:
      // read on after it; anything else, or the end of the text or document:
      // the last).  Every lane holds the same position and answer; offsets
      // are from the window's end.
      if (wave == 0) {
        const uint8_t* base = w.text + (w0 + PT_WIN);
        int64_t lim = n;
        if (BATCH) {
          int lo = 0, hi = w.n_docs;
          while (lo < hi) {
            int mid = (lo + hi) >> 1;
            if (w.doc_off[mid] < w0 + PT_WIN) lo = mid + 1;
            else hi = mid;
          }
          if (lo < w.n_docs && w.doc_off[lo] < lim) lim = w.doc_off[lo];
        }
        const uint32_t end = (uint32_t)(lim - (w0 + PT_WIN));
        uint32_t pos = 0, res = 2u;
        while (pos < end && (base[pos] & 0xC0u) == 0x80u) ++pos;
#pragma unroll 1
        while (res == 2u) {
          uint32_t first = 16u;
#pragma unroll 4
          for (int k = 15; k >= 0; --k) {
            const uint32_t p = pos + 16u * (uint32_t)lane + (uint32_t)k;
            const uint32_t b = p < end ? (uint32_t)base[p] : 0u;  // (the end counts as a stop)
            if (b != 0x20u && b != 0x09u && b != 0x0Bu && b != 0x0Cu) first = (uint32_t)k;
          }
          const uint64_t m = __ballot(first < 16u);
          if (m == 0ull) {
            pos += 16u * 64u;
            continue;
          }
          const int src = __builtin_ctzll(m);
          const uint32_t p = pos + 16u * (uint32_t)src + (uint32_t)__builtin_amdgcn_readlane((int)first, src);
          if (p >= end) {
            res = 1u;
            break;
          }
          const uint32_t avail = end - p < 4u ? end - p : 4u;
          auto at = [&](uint32_t k) -> uint32_t { return k < avail ? (uint32_t)base[p + k] : 0u; };
          uint32_t cp = 0;
          const uint32_t len = decode_sel(at(0), at(1), at(2), at(3), avail, cp);
          const uint32_t c = len == 0u ? (uint32_t)C_O : code_cls(char_code_sel<PAT>(sh.ph.a.cls, cp));
          if (len == 0u) res = 1u;  // invalid input; reported elsewhere
          else if (c == C_NL) res = 0u;
          else if (c != C_WS) res = 1u;
          else pos = p + len;
        }
        if (lane == 0) sh.ws_res = res;
      }
      __syncthreads();
      if (sh.ws_res == 1u && tid == pend / PT_BPT) flags |= 1u << (pend % PT_BPT);
    }
  }
  const bool last = t == n_tiles - 1;
  if (IGN) {
    // ignore_merges: a piece that is a vocabulary entry is that entry's ID
    // (Sec. 4.2: the vocabulary is probed first and the merge loop skipped).
    // Pieces are numbered by a block scan (their starts go to sh.ustart until
    // the unit scan), every piece that ends inside the tile is probed, and no
    // junction cut may split a piece found in the vocabulary.  The pieces that
    // cross the tile's edges are not cut at all: the next tile encodes the
    // last one whole, as its incoming unit, and probes it there.
    const uint32_t pc = __popc(flags);
    const uint32_t pinc = wave_incl_sum(pc);
    __syncthreads();
    if (lane == 63) sh.wave_tot[wave] = pinc;
    __syncthreads();
    uint32_t pw = 0, pm = 0;
    for (int v = 0; v < PT_THREADS / 64; ++v) {
      if (v < wave) pw += sh.wave_tot[v];
      pm += sh.wave_tot[v];
    }
    {
      uint32_t k = pw + pinc - pc;
#pragma unroll 1
      for (int j = 0; j < PT_BPT; ++j)
        if ((flags >> j) & 1u) sh.ustart[k++] = (uint16_t)(qb + j);
    }
    if (tid == 0) sh.ustart[pm] = (uint16_t)(last ? n - w0 : 0xFFFFu);  // end of the last piece, if known
    __syncthreads();
#pragma unroll 1
    for (uint32_t k = (uint32_t)tid; k < pm; k += PT_THREADS) {
      const uint32_t a = sh.ustart[k], e = sh.ustart[k + 1];
      if (e == 0xFFFFu) continue;
      const uint32_t L = e - a;
      if (L < 2u || L > tb.vmax) continue;
      const uint32_t id = piece_find(tb, sh.buf, (int64_t)a, L, [&](uint32_t j) -> uint32_t { return sh.buf[PT_PAD + a + j]; });
      if (id == DICT_NONE) continue;
      w.stage[w0 + a] = id;
      atomicOr(&sh.whole[a >> 5], 1u << (a & 31u));
      for (uint32_t q = a + 1; q < e; ++q) atomicOr(&sh.ph.a.nocut[q >> 5], 1u << (q & 31u));
    }
    // the incoming piece's tail and the tile's last piece
    const uint32_t first = pm > 0 ? sh.ustart[0] : (uint32_t)(PT_HALO + PT_OWN);
    const uint32_t lastp = pm > 0 ? sh.ustart[pm - 1] : (uint32_t)PT_HALO;
    uint32_t mask = 0;
#pragma unroll
    for (int j = 0; j < PT_BPT; ++j) {
      const uint32_t q = (uint32_t)(qb + j);
      const bool own = q >= (uint32_t)PT_HALO && q < (uint32_t)(PT_HALO + PT_OWN);
      if (own && ((t > 0 && q < first) || (!last && q > lastp))) mask |= 1u << j;
    }
    if (mask) atomicOr(&sh.ph.a.nocut[qb >> 5], mask << (qb & 31));
    __syncthreads();
  }
  TT_PHASE(22);
  if (SEG) {
    // BPE segments: add the byte positions inside pieces that no merge spans
    // (q is not a piece start, so q - 1 lies in the same piece)
    const uint32_t* bwp = reinterpret_cast<const uint32_t*>(&sh.buf[PT_PAD + qb - 4]);
    const uint64_t bb = bwp[0] | ((uint64_t)bwp[1] << 32);  // bytes of positions qb - 4 .. qb + 3
#pragma unroll
    for (int j = 0; j < PT_BPT; ++j) {
      const int q = qb + j;
      const uint32_t key = (uint32_t)((bb >> (8 * (j + 3))) & 0xFFFFull);  // (b[q-1], b[q]) as b[q-1] | b[q] << 8
      const uint32_t k2 = ((key & 255u) << 8) | (key >> 8);
      const bool joined = (sh.ph.a.join[k2 >> 5] >> (k2 & 31u)) & 1u;
      const bool eligible = q >= PT_HALO && q < PT_HALO + PT_OWN && inside(q) && inside(q - 1) &&
                            !(flags & (1u << j)) && !(cr(j) & CODE_DOCSTART) &&
                            !(IGN && ((sh.ph.a.nocut[q >> 5] >> (q & 31)) & 1u));
      if (eligible && !joined) flags |= 1u << j;
    }
  }

  TT_PHASE(5);
  TT_PHASE_BY(24 + wave, lane == 0);
  // ---- units: block scan of the start flags --------------------------------
  const uint32_t cnt = __popc(flags);
  const uint32_t inc = wave_incl_sum(cnt);
  __syncthreads();
  if (lane == 63) sh.wave_tot[wave] = inc;
  __syncthreads();
  uint32_t wpre = 0, m = 0;
  for (int v = 0; v < PT_THREADS / 64; ++v) {
    if (v < wave) wpre += sh.wave_tot[v];
    m += sh.wave_tot[v];
  }
  wpre = wave_uniform(wpre);
  m = wave_uniform(m);
  const uint32_t texcl = wpre + inc - cnt;  // unit starts before this thread's positions

  if (MODE == 0) {
    // split export: the tile's piece offsets go straight to their place
    const uint32_t prefix = place_tile(w, sh, t, m, tile_bad, tid, lane, wave);
    uint32_t k = prefix + texcl;
#pragma unroll 1
    for (int j = 0; j < PT_BPT; ++j)
      if (((flags >> j) & 1u) && k < (uint32_t)n) w.out_ids[k++] = (int32_t)(w0 + qb + j);
    return;
  }

  TT_PHASE(11);
  // the tile's last unit start, published before this block waits on anything
  if (m == 0) {
    if (tid == 0) st_word(&w.tile_last[t], ((uint64_t)w.epoch << 32) | NO_START);
  } else if (cnt != 0u && texcl + cnt == m) {
    st_word(&w.tile_last[t], ((uint64_t)w.epoch << 32) | (uint32_t)(w0 + qb + 31 - __builtin_clz(flags)));
  }
  {
    uint32_t k = texcl;
#pragma unroll 1
    for (int j = 0; j < PT_BPT; ++j)
      if ((flags >> j) & 1u) sh.ustart[k++] = (uint16_t)(qb + j);
  }
  if (tid == 0) sh.ustart[m] = (uint16_t)(last ? n - w0 : 0);

  // The units this tile encodes: its own units but the last (whose end lies
  // in a later tile), all of them in the last tile, and the incoming unit
  // that ends at its first unit start.
  const bool has_inc = t > 0 && (m > 0 || last);
  const uint32_t m_proc = last ? m : (m > 0 ? m - 1 : 0);
  __syncthreads();
  const uint32_t e_inc = wave_uniform(m > 0 ? (uint32_t)(w0 + sh.ustart[0]) : (uint32_t)n);
  auto byte_abs = [&](uint32_t p) -> uint32_t {
    const int64_t q = (int64_t)p - w0;
    return (q >= -PT_PAD && q < PT_WIN + 16) ? (uint32_t)sh.buf[PT_PAD + q] : (uint32_t)w.text[p];
  };
  // The incoming unit starts at the last unit start of the nearest earlier
  // tile that has one (usually the previous tile).  Only the thread that
  // dispatches it waits for that word; the others dispatch their own units
  // meanwhile.  (Only invalid input, whose text starts with a continuation
  // byte, leaves no unit start before the tile; its output is discarded.)
  TT_PHASE(12);
  uint32_t sp_own = 0;
  if (has_inc && (uint32_t)tid == m_proc % (uint32_t)PT_THREADS) {
    uint32_t found = NO_START;
    for (int64_t j = (int64_t)t - 1; j >= 0; --j) {
      const uint64_t x = wait_word(&w.tile_last[j], w.epoch);
      if ((uint32_t)x != NO_START) {
        found = (uint32_t)x;
        break;
      }
    }
    sh.s_prev = found;
    sp_own = found != NO_START ? found : 0u;
    TT_PHASE_BY(20, true);
  }
  auto inc_byte_own = [&](uint32_t j) -> uint32_t { return byte_abs(sp_own + j); };
  auto inc_out_own = [&](uint32_t j, uint32_t id) { w.stage[sp_own + j] = id; };

  // ---- BPE dispatch ---------------------------------------------------------
  // Units of one or two bytes are finished here, and so are units of up to 24
  // bytes found in the whole-unit dictionaries.  Other units of 3..16 bytes go to
  // one thread each, counting-sorted by length, so that the threads of a wave
  // hold units of similar length (a wave runs as long as its longest unit).
  // Units of 17..WAVE_MAX bytes go to one wave each, longest first, to the
  // waves as they become free (no block barrier between the two engines), and
  // longer units to the whole block.
  constexpr int UPT = (PT_OWN + 1 + PT_THREADS - 1) / PT_THREADS;  // units per thread
  const uint32_t U = m_proc + (has_inc ? 1u : 0u);
  uint32_t mine[UPT];  // thread and wave units: (length << 16) | position within its length class
#pragma unroll
  for (int r = 0; r < UPT; ++r) {
    mine[r] = 0;
    const uint32_t u = (uint32_t)(tid + r * PT_THREADS);
    if (u >= U) continue;
    const bool inc_u = u == m_proc;
    const uint32_t a = inc_u ? 0u : sh.ustart[u];
    const uint32_t L = inc_u ? e_inc - sp_own : sh.ustart[u + 1] - a;
    if (IGN) {
      // a piece found in the vocabulary (its ID was staged at its first byte);
      // the incoming unit is a whole piece and is probed here
      uint32_t id = DICT_NONE;
      if (!inc_u && ((sh.whole[a >> 5] >> (a & 31u)) & 1u)) {
        id = w.stage[w0 + a];
      } else if (inc_u && L >= 2u && L <= tb.vmax) {
        id = piece_find(tb, sh.buf, (int64_t)sp_own - w0, L, [&](uint32_t j) -> uint32_t { return inc_byte_own(j); });
      }
      if (id != DICT_NONE) {
        if (inc_u) {
          inc_out_own(0, id);
          sh.inc_cnt = 1;
        } else {
          sh.ph.b.tok[a] = id;
          sh.ucnt[u] = 1;
        }
        continue;
      }
    }
    if (L <= 2u) {
      const uint32_t b0 = inc_u ? inc_byte_own(0) : sh.buf[PT_PAD + a];
      uint32_t c = 1, t0 = b0, t1 = 0;
      if (L == 2u) {
        const uint32_t b1 = inc_u ? inc_byte_own(1) : sh.buf[PT_PAD + a + 1];
        const uint32_t r2 = tb.pair0[(b0 << 8) | b1];
        if (r2 != RANK_INF) {
          t0 = 256u + r2;
        } else {
          c = 2;
          t1 = b1;
        }
      }
      if (inc_u) {
        inc_out_own(0, t0);
        if (c == 2) inc_out_own(1, t1);
        sh.inc_cnt = c;
      } else {
        sh.ph.b.tok[a] = t0;
        if (c == 2) sh.ph.b.tok[a + 1] = t1;
        sh.ucnt[u] = (uint16_t)c;
      }
    } else {
      // units of 3..24 bytes: the whole-unit dictionaries first.  Their bytes
      // are in the window (an incoming unit this short ends at the tile's
      // first unit start, so it starts at least PT_HALO - 24 bytes into it).
      uint32_t found = DICT_NONE;
      const int64_t aw = inc_u ? (int64_t)sp_own - w0 : (int64_t)a;
      if (L <= (uint32_t)DICT2_MAX && aw >= 0 && aw + DICT2_MAX + 4 <= PT_WIN + 16) {
        if (L <= (uint32_t)DICT_MAX) {
          uint32_t kw[3];
          unit_words(sh.buf, (uint32_t)aw, L, kw);
          found = dict_find(tb.dict, tb.dnb, kw[0], kw[1], kw[2], L);
        } else {
          uint32_t kw[6];
          unit_words(sh.buf, (uint32_t)aw, L, kw);
          found = dict2_find(tb.dict2, tb.dnb2, kw, L);
        }
      }
      if (found != DICT_NONE) {
        if (inc_u) {
          inc_out_own(0, found);
          sh.inc_cnt = 1;
        } else {
          sh.ph.b.tok[a] = found;
          sh.ucnt[u] = 1;
        }
      } else if (L <= (uint32_t)SMALL_MAX) {
        mine[r] = (L << 16) | atomicAdd(&sh.hist[L], 1u);
      } else if (L <= (uint32_t)WAVE_MAX) {
        mine[r] = (L << 16) | atomicAdd(&sh.hmed[med_class(L)], 1u);
      } else {
        sh.big[atomicAdd(&sh.n_big, 1u)] = inc_u ? U_INCOMING : (uint16_t)u;
      }
    }
  }
  __syncthreads();
  const uint32_t s_prev = wave_uniform(has_inc && sh.s_prev != NO_START ? sh.s_prev : 0u);
  const uint32_t L_inc = has_inc ? e_inc - s_prev : 0u;
  auto inc_byte = [&](uint32_t j) -> uint32_t { return byte_abs(s_prev + j); };
  auto inc_out = [&](uint32_t j, uint32_t id) { w.stage[s_prev + j] = id; };
  TT_PHASE(13);
  // where each length (class) starts: a wave scan over the counts (wave 0 for
  // the thread units, wave 1 for the wave units)
  if (wave == 0) {
    const bool in = lane >= 3 && lane <= SMALL_MAX;
    const uint32_t c = in ? sh.hist[lane] : 0u;
    const uint32_t incl = wave_incl_sum(c);
    if (in) sh.hist[lane] = incl - c;
    if (lane == SMALL_MAX) sh.n_small = incl;
  } else if (wave == 1) {
    const bool in = lane < MED_CLASSES;
    const uint32_t c = in ? sh.hmed[lane] : 0u;
    const uint32_t incl = wave_incl_sum(c);
    if (in) sh.hmed[lane] = incl - c;
    if (lane == MED_CLASSES - 1) sh.n_med = incl;
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < UPT; ++r) {
    if (mine[r] == 0) continue;
    const uint32_t u = (uint32_t)(tid + r * PT_THREADS);
    const uint16_t e = u == m_proc ? U_INCOMING : (uint16_t)u;
    const uint32_t L = mine[r] >> 16, pos = mine[r] & 0xFFFFu;
    if (L <= (uint32_t)SMALL_MAX) sh.ph.b.small[sh.hist[L] + pos] = e;
    else sh.med[sh.hmed[med_class(L)] + pos] = e;
  }
  __syncthreads();
  TT_PHASE(14);
  const uint32_t n_small = wave_uniform(sh.n_small), n_med = wave_uniform(sh.n_med);

  TT_PHASE(6);
  // thread per unit, on the first TH_THREADS threads
  if (tid < TH_THREADS) {
    uint32_t* rk = &sh.ph.b.rk[0][tid];
#pragma unroll 1
    for (uint32_t i = tid; i < n_small; i += TH_THREADS) {
      const uint32_t u = sh.ph.b.small[i];
      const bool inc_u = u == U_INCOMING;
      // a unit's own window slots hold its tokens while it is encoded (the
      // incoming unit's are in inc_ids); one call site, so that a wave does
      // not run the merge loop twice when it holds the incoming unit
      const uint32_t a = inc_u ? 0u : sh.ustart[u];
      const uint32_t L = inc_u ? L_inc : sh.ustart[u + 1] - a;
      uint32_t* ids = inc_u ? sh.inc_ids : &sh.ph.b.tok[a];
      for (uint32_t j = 0; j < L; ++j) ids[j] = inc_u ? inc_byte(j) : (uint32_t)sh.buf[PT_PAD + a + j];
      const uint32_t c = bpe_thread(L, ids, rk, tb);
      if (inc_u) {
        for (uint32_t j = 0; j < c; ++j) inc_out(j, ids[j]);
        sh.inc_cnt = c;
      } else {
        sh.ucnt[u] = (uint16_t)c;
      }
    }
  }

  // wave per unit: the units are taken longest first from a shared queue,
  // each by the next wave that is free (the waves with thread work join when
  // it is done), so that no wave runs two long units while another idles
  {
#pragma unroll 1
    for (;;) {
      // all 64 lanes add one (no branch on the lane before the broadcast,
      // which would make the loop exit divergent), so a wave's grab moves the
      // counter by 64 and lane 0 reads a multiple of 64
      const uint32_t i = wave_uniform(atomicAdd(&sh.med_next, 1u)) / 64u;
      if (i >= n_med) break;
      const uint32_t u = wave_uniform(sh.med[i]);
      const bool inc_u = u == U_INCOMING;
      const uint32_t a = inc_u ? 0u : sh.ustart[u];
      const uint32_t L = inc_u ? L_inc : sh.ustart[u + 1] - a;
      if (!(IGN && SPANS) && L <= 32u) {
        // the queue is in 8-byte length classes, longest first, and 32 bytes
        // end a class, so every unit left has at most 32 bytes too: take the
        // next one as well, one unit per half wave (not in the rarely used
        // ignore_merges span export, which it would push into spills)
        const uint32_t i2 = wave_uniform(atomicAdd(&sh.med_next, 1u)) / 64u;
        if (i2 < n_med) {
          const uint32_t u2 = wave_uniform(sh.med[i2]);
          const bool inc2 = u2 == U_INCOMING;
          const uint32_t a2 = inc2 ? 0u : sh.ustart[u2];
          const uint32_t L2 = inc2 ? L_inc : sh.ustart[u2 + 1] - a2;
          auto by2 = [&](uint32_t hf, uint32_t j) -> uint32_t {
            const bool in = hf ? inc2 : inc_u;
            return in ? inc_byte(j) : (uint32_t)sh.buf[PT_PAD + (hf ? a2 : a) + j];
          };
          auto ot2 = [&](uint32_t hf, uint32_t j, uint32_t id) {
            if (hf ? inc2 : inc_u) inc_out(j, id);
            else sh.ph.b.tok[(hf ? a2 : a) + j] = id;
          };
          const uint32_t c2 = bpe_pair32(L, L2, by2, tb, ot2);
          if (lane == 0) {
            if (inc_u) sh.inc_cnt = c2 & 0xFFFFu;
            else sh.ucnt[u] = (uint16_t)(c2 & 0xFFFFu);
            if (inc2) sh.inc_cnt = c2 >> 16;
            else sh.ucnt[u2] = (uint16_t)(c2 >> 16);
          }
          continue;
        }
      }
      auto by = [&](int j) -> uint32_t {
        return inc_u ? inc_byte((uint32_t)j) : (uint32_t)sh.buf[PT_PAD + a + (uint32_t)j];
      };
      auto ot = [&](int j, uint32_t id) {
        if (inc_u) inc_out((uint32_t)j, id);
        else sh.ph.b.tok[a + (uint32_t)j] = id;
      };
      uint32_t* scr = sh.ph.b.x.wscr[wave];
      const uint32_t c = L <= 64u ? bpe_wave(L, by, tb, ot) : bpe_wave2(L, by, tb, scr, ot);
      if (lane == 0) {
        if (inc_u) sh.inc_cnt = c;
        else sh.ucnt[u] = (uint16_t)c;
      }
    }
  }
  __syncthreads();

  TT_PHASE(7);
  // ---- BPE, whole block per longer unit ------------------------------------
  // (rare in text: rows in LDS up to ROWS_LDS bytes, else in global scratch
  // at the unit's byte offset; there the selection masks of a unit of L > 64
  // bytes at byte s take words [s/16, s/16 + L/64 + 2), which never reach the
  // next unit's)
  const uint32_t n_big = sh.n_big;
#pragma unroll 1
  for (uint32_t i = 0; i < n_big; ++i) {
    const uint32_t u = sh.big[i];
    const bool inc_u = u == U_INCOMING;
    const uint32_t a = inc_u ? 0u : sh.ustart[u];
    const uint32_t L = inc_u ? L_inc : sh.ustart[u + 1] - a;
    const uint64_t s0 = inc_u ? (uint64_t)s_prev : (uint64_t)(w0 + a);
    uint32_t *I0, *I1, *R0, *R1;
    uint64_t* sel;
    if (L <= (uint32_t)ROWS_LDS) {
      auto& rw = sh.ph.b.x.rows;
      I0 = rw.I0;
      I1 = rw.I1;
      R0 = rw.R0;
      R1 = rw.R1;
      sel = rw.sel;
    } else {
      uint32_t* sc = w.scratch;
      const uint64_t nn = (uint64_t)n;
      I0 = sc + s0;
      I1 = sc + nn + s0;
      R0 = sc + 2 * nn + s0;
      R1 = sc + 3 * nn + s0;
      sel = reinterpret_cast<uint64_t*>(sc + 4 * nn) + s0 / 16;
    }
    uint32_t c;
    if (inc_u) {
      c = bpe_rows<PT_THREADS / 64>(L, inc_byte, tb, I0, I1, R0, R1, sel, sh.rows, inc_out);
    } else {
      c = bpe_rows<PT_THREADS / 64>(
          L, [&](uint32_t j) -> uint32_t { return sh.buf[PT_PAD + a + j]; }, tb, I0, I1, R0, R1, sel, sh.rows,
          [&](uint32_t j, uint32_t id) { sh.ph.b.tok[a + j] = id; });
    }
    if (tid == 0) {
      if (inc_u) sh.inc_cnt = c;
      else sh.ucnt[u] = (uint16_t)c;
    }
    __syncthreads();
  }

  TT_PHASE(8);
  // ---- output: the tile's tokens, in order, at their place --------------------
  uint32_t csum = 0;
#pragma unroll 1
  for (int j = 0; j < PT_BPT; ++j) {
    const uint32_t k = (uint32_t)(tid * PT_BPT + j);
    csum += k < m_proc ? sh.ucnt[k] : 0u;
  }
  const uint32_t cinc = wave_incl_sum(csum);
  if (lane == 63) sh.wave_tot[wave] = cinc;
  __syncthreads();
  uint32_t cpre = 0, ctot = 0;
  for (int v = 0; v < PT_THREADS / 64; ++v) {
    if (v < wave) cpre += sh.wave_tot[v];
    ctot += sh.wave_tot[v];
  }
  {
    uint32_t o = cpre + cinc - csum;
#pragma unroll 1
    for (int j = 0; j < PT_BPT; ++j) {
      const uint32_t k = (uint32_t)(tid * PT_BPT + j);
      if (k < m_proc) {
        sh.ph.b.uoff[k] = (uint16_t)o;
        o += sh.ucnt[k];
      }
    }
  }
  const uint32_t inc_cnt = has_inc ? sh.inc_cnt : 0u;
  // (place_tile ends with a barrier, which also publishes uoff to the block)
  const uint32_t prefix = place_tile(w, sh, t, inc_cnt + ctot, tile_bad, tid, lane, wave,
                                     SPANS ? w.tile_cagg : nullptr, SPANS ? sh.ctile : 0u);
  TT_PHASE(9);
  // Valid input gives every tile a disjoint byte range and at most one output
  // per byte, so every output index is below n.  Invalid input (whose output
  // is discarded) can break that; the bound keeps it inside the buffer.
  const uint32_t lim = (uint32_t)n;
  int32_t* __restrict__ out = w.out_ids;
  const int32_t* __restrict__ ext = tb.ext_id;
  auto ext_of = [&](uint32_t v) -> int32_t { return v < tb.n_ids ? ext[v] : -1; };
  // (narrow IDs: single requests of tt_encode only)
  uint16_t* __restrict__ out16 = (SPANS || BATCH) ? nullptr : w.out16;
  uint8_t* __restrict__ out_hi = (SPANS || BATCH) ? nullptr : w.out_hi;
  for (uint32_t i = (uint32_t)tid; i < inc_cnt; i += PT_THREADS) {
    if (prefix + i >= lim) continue;
    const int32_t v = ext_of(w.stage[s_prev + i]);
    if (out16) {
      out16[prefix + i] = (uint16_t)v;
      if (out_hi) out_hi[prefix + i] = (uint8_t)((uint32_t)v >> 16);
    } else {
      out[prefix + i] = v;
    }
  }
  const uint32_t obase = prefix + inc_cnt;
  // Token o of unit k sits at position ustart[k] + o, so the tokens of a
  // wave's positions go to one contiguous range of the output, in position
  // order.  Without span export (which reads tok[] again) each wave first
  // packs its tokens at the front of its own part of tok[] and then writes
  // the range with consecutive lanes on consecutive words: whole lines, which
  // matters most when the output is pinned host memory.
  uint32_t before = texcl;  // unit starts at or before position q
  int32_t val[PT_BPT];
  uint32_t at_of[PT_BPT];
  uint32_t has = 0;
#pragma unroll
  for (int j = 0; j < PT_BPT; ++j) {
    const int q = qb + j;
    const bool st = (flags >> j) & 1u;
    before += st ? 1u : 0u;
    val[j] = 0;
    at_of[j] = 0;
    if (before == 0u || before - 1u >= m_proc) continue;
    const uint32_t k = before - 1u;
    const uint32_t o = (uint32_t)q - sh.ustart[k];
    const uint32_t at = obase + sh.ph.b.uoff[k] + o;
    if (o < sh.ucnt[k] && at < lim) {
      val[j] = ext_of(sh.ph.b.tok[q]);
      at_of[j] = at;
      has |= 1u << j;
    }
    if (BATCH && st && sh.dstart[PT_PAD + q]) {
      w.unit_tile[w0 + q] = t;
      w.unit_pos[w0 + q] = inc_cnt + sh.ph.b.uoff[k];
    }
  }
  if (SPANS) {
#pragma unroll
    for (int j = 0; j < PT_BPT; ++j)
      if ((has >> j) & 1u) out[at_of[j]] = val[j];
  } else {
    const uint32_t mine = (uint32_t)__builtin_popcount(has);
    const uint32_t incl = wave_incl_sum(mine);
    const uint32_t n_wave = (uint32_t)__builtin_amdgcn_readlane((int)incl, 63);
    const uint64_t holders = __ballot(mine != 0u);
    // the wave's first output index (the lowest lane holding a token, its
    // lowest position with one)
    const uint32_t first = (has & 1u) ? at_of[0] : (has & 2u) ? at_of[1] : (has & 4u) ? at_of[2] : at_of[3];
    const uint32_t base = holders ? (uint32_t)__builtin_amdgcn_readlane((int)first, (int)__builtin_ctzll(holders)) : 0u;
    uint32_t* pack = &sh.ph.b.tok[wave * 64 * PT_BPT];
    __syncthreads();  // every read of tok[] above is done
    uint32_t r = incl - mine;
#pragma unroll
    for (int j = 0; j < PT_BPT; ++j)
      if ((has >> j) & 1u) pack[r++] = (uint32_t)val[j];
    __syncthreads();
    // (valid text: the wave's indices are exactly base .. base + n_wave - 1)
    if (out16) {
      for (uint32_t i = (uint32_t)lane; i < n_wave; i += 64)
        if (base + i < lim) out16[base + i] = (uint16_t)pack[i];
      if (out_hi)
        for (uint32_t i = (uint32_t)lane; i < n_wave; i += 64)
          if (base + i < lim) out_hi[base + i] = (uint8_t)(pack[i] >> 16);
    } else {
      for (uint32_t i = (uint32_t)lane; i < n_wave; i += 64)
        if (base + i < lim) out[base + i] = (int32_t)pack[i];
    }
  }
  if (BATCH && tid == 0 && has_inc) {
    w.unit_tile[s_prev] = t;
    w.unit_pos[s_prev] = 0;
  }
  if (SPANS) {
    // byte start of every token: its unit's start plus the byte lengths of the
    // unit's earlier tokens (byte-level BPE fixes every token's length)
    auto len_of = [&](uint32_t v) -> uint32_t { return v < tb.n_ids ? tb.tok_len[v] : 0u; };
    // the incoming unit's tokens, PT_THREADS at a time
    uint32_t carry = 0;
#pragma unroll 1
    for (uint32_t base = 0; base < inc_cnt; base += PT_THREADS) {
      const uint32_t i = base + (uint32_t)tid;
      const uint32_t len = i < inc_cnt ? len_of(w.stage[s_prev + i]) : 0u;
      const uint32_t wi = wave_incl_sum(len);
      if (lane == 63) sh.cwave[wave] = wi;
      __syncthreads();
      uint32_t pre = 0, tot = 0;
      for (int v = 0; v < PT_THREADS / 64; ++v) {
        if (v < wave) pre += sh.cwave[v];
        tot += sh.cwave[v];
      }
      if (i < inc_cnt && prefix + i < lim) w.out_spans[4 * (size_t)(prefix + i)] = (int32_t)(s_prev + carry + pre + wi - len);
      carry += tot;
      __syncthreads();
    }
    // the tile's own units: a scan over the window positions, restarted at
    // every unit start, of the lengths of the tokens held there
    constexpr uint32_t HEAD = 0x80000000u;
    auto seg_add = [](uint32_t a, uint32_t b) -> uint32_t {
      return (b & HEAD) ? b : ((a & HEAD) | ((a + b) & ~HEAD));
    };
    uint32_t e[PT_BPT];
    uint32_t agg = 0;
    {
      uint32_t bf = texcl;
#pragma unroll
      for (int j = 0; j < PT_BPT; ++j) {
        const int q = qb + j;
        const uint32_t hd = (flags >> j) & 1u;
        bf += hd;
        const uint32_t k = bf - 1u;
        const bool tokq = bf != 0u && k < m_proc && (uint32_t)q - sh.ustart[k] < sh.ucnt[k];
        e[j] = tokq ? len_of(sh.ph.b.tok[q]) : 0u;
        agg = seg_add(agg, (hd ? HEAD : 0u) | e[j]);
      }
    }
    const uint32_t winc = wave_incl_scan(agg, lane, seg_add);
    if (lane == 63) sh.cwave[wave] = winc;
    uint32_t st = (uint32_t)__shfl_up((int)winc, 1, 64);
    if (lane == 0) st = 0;
    __syncthreads();
    uint32_t wpre = 0;
    for (int v = 0; v < wave; ++v) wpre = seg_add(wpre, sh.cwave[v]);
    st = seg_add(wpre, st);
    uint32_t bf = texcl;
#pragma unroll
    for (int j = 0; j < PT_BPT; ++j) {
      const int q = qb + j;
      const uint32_t hd = (flags >> j) & 1u;
      bf += hd;
      const uint32_t k = bf - 1u;
      if (bf != 0u && k < m_proc) {
        const uint32_t o = (uint32_t)q - sh.ustart[k];
        const uint32_t at = obase + sh.ph.b.uoff[k] + o;
        const uint32_t within = hd ? 0u : (st & ~HEAD);
        if (o < sh.ucnt[k] && at < lim) w.out_spans[4 * (size_t)at] = (int32_t)(w0 + sh.ustart[k] + within);
      }
      st = seg_add(st, (hd ? HEAD : 0u) | e[j]);
    }
    // non-continuation bytes before every 4-byte word of the tile's own range
    // (and before the end of the text), for the character spans
    const int q0 = tid * PT_BPT;
    const int64_t p0 = w0 + q0;
    const uint32_t nc = own_noncont(*reinterpret_cast<const uint32_t*>(&sh.buf[PT_PAD + q0]), q0, p0);
    const uint32_t nci = wave_incl_sum(nc);
    __syncthreads();  // (the scan above has read sh.cwave)
    if (lane == 63) sh.cwave[wave] = nci;
    __syncthreads();
    uint32_t c_excl = nci - nc;
    for (int v = 0; v < wave; ++v) c_excl += sh.cwave[v];
    if (q0 >= PT_HALO && q0 < PT_HALO + PT_OWN && p0 < n) w.ccount[p0 >> 2] = sh.cbase + c_excl;
    if (last && tid == 0 && (n & 3) == 0) w.ccount[n >> 2] = sh.cbase + sh.ctile;
  }
#ifdef TT_PHASE_STAMPS
  __syncthreads();
  TT_PHASE(10);
#endif
}

namespace {
template <int PAT>
hipError_t launch_pat(const Work& w, const DevTables& tb, int mode, bool batch, bool ignore, hipStream_t s) {
  dim3 grid(w.n_tiles), block(PT_THREADS);
#define TT_TILE(B, M, I) hipLaunchKernelGGL((tile_kernel<PAT, B, M, I>), grid, block, 0, s, w, tb)
  if (mode == 0) {
    if (ignore) return hipErrorInvalidValue;  // the split export has no model stage
    if (batch) TT_TILE(true, 0, false);
    else TT_TILE(false, 0, false);
  } else if (mode == 1) {
    if (batch && ignore) TT_TILE(true, 1, true);
    else if (batch) TT_TILE(true, 1, false);
    else if (ignore) TT_TILE(false, 1, true);
    else TT_TILE(false, 1, false);
  } else {
    if (batch) return hipErrorInvalidValue;  // span export is for single requests
    if (ignore) TT_TILE(false, 2, true);
    else TT_TILE(false, 2, false);
  }
#undef TT_TILE
  return hipGetLastError();
}
}  // namespace

hipError_t launch_tile(const Work& w, const DevTables& tb, int pattern, int mode, bool ignore, hipStream_t s) {
  const bool batch = w.doc_off != nullptr;
  switch (pattern) {
    case TT_PATTERN_GPT2: return launch_pat<TT_PATTERN_GPT2>(w, tb, mode, batch, ignore, s);
    case TT_PATTERN_CL100K: return launch_pat<TT_PATTERN_CL100K>(w, tb, mode, batch, ignore, s);
    case TT_PATTERN_O200K: return launch_pat<TT_PATTERN_O200K>(w, tb, mode, batch, ignore, s);
    case TT_PATTERN_DEEPSEEK: return launch_pat<TT_PATTERN_DEEPSEEK>(w, tb, mode, batch, ignore, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace tt

#ifdef TT_PHASE_STAMPS
// The phase stamps of the first n_tiles tiles of the last call (n_tiles *
// TT_PHASE_SLOTS words, tile-major) into out (host memory).  Diagnostic build
// only; returns TT_OK, TT_ERR_BAD_ARG or TT_ERR_HIP.
extern "C" int tt_phase_stamps(unsigned long long* out, int n_tiles) {
  if (!out || n_tiles < 0 || n_tiles > tt::TT_PHASE_TILES) return TT_ERR_BAD_ARG;
  const hipError_t e = hipMemcpyFromSymbol(out, HIP_SYMBOL(tt::tt_phase_buf),
                                           (size_t)n_tiles * tt::TT_PHASE_SLOTS * sizeof(unsigned long long), 0,
                                           hipMemcpyDeviceToHost);
  return e == hipSuccess ? TT_OK : TT_ERR_HIP;
}
#endif
