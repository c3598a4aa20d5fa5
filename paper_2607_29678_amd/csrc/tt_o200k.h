// The o200k-style pattern (Sec. 4.1: the o200k lineage adds a case-boundary
// rule and treats Unicode marks specially).  Its alternatives, in order:
//   P1  [^\r\n\p{L}\p{N}]? [Lu Lt Lm Lo M]* [Ll Lm Lo M]+ CT?
//   P2  [^\r\n\p{L}\p{N}]? [Lu Lt Lm Lo M]+ [Ll Lm Lo M]* CT?
//   P3  \p{N}{1,3}
//   P4  U+0020? [^\s\p{L}\p{N}]+ [\r\n/]*
//   P5  \s*[\r\n]+      P6  \s+(?!\S)      P7  \s+
// where CT is the case-insensitive contraction 's 't 're 've 'm 'll 'd.
//
// The piece boundaries are not all local here: whether an upper-case run
// keeps its last characters depends on what follows the whole run, and marks
// belong to letter runs and to symbol runs alike.  So the tile kernel finds
// the positions where the pattern resets for every left context (the
// synchronizing transitions below, the same sets that certify splices in
// incremental repair) and resolves the pieces between two such positions by
// running the pattern's alternatives from the first one: one thread walks one
// segment, piece by piece, over the window in LDS.
#pragma once

#include "tt_internal.h"

namespace tt {

// Classes of the o200k-style pattern (4 bits of a window code).
enum : uint32_t {
  O2_O = 0,    // other
  O2_UP = 1,   // Lu, Lt: only in the upper-case letter set
  O2_LO = 2,   // Ll: only in the lower-case letter set
  O2_BO = 3,   // Lm, Lo: in both letter sets
  O2_MK = 4,   // M: in both letter sets and in the "not letter, not number" sets
  O2_N = 5,    // \p{N}
  O2_WS = 6,   // \s except CR and LF
  O2_NL = 7,   // CR, LF
  O2_NONE = 15 // continuation byte, or outside the text
};

__host__ __device__ constexpr bool o2_letter(uint32_t c) { return c == O2_UP || c == O2_LO || c == O2_BO; }
__host__ __device__ inline bool o2_ub(uint32_t c) { return c == O2_UP || c == O2_BO || c == O2_MK; }
__host__ __device__ inline bool o2_lb(uint32_t c) { return c == O2_LO || c == O2_BO || c == O2_MK; }
__host__ __device__ inline bool o2_oset(uint32_t c) { return c == O2_O || c == O2_MK; }
__host__ __device__ inline bool o2_space(uint32_t c) { return c == O2_WS || c == O2_NL; }

// Class of a code point from the probed 4-bit table (levels l1, l2; host
// arrays, or the copy a block keeps in LDS).
template <class P>
__host__ __device__ inline uint32_t o2_table_class(P l1, P l2, uint32_t cp) {
  if (cp == 10u || cp == 13u) return O2_NL;
  const uint32_t blk = l1[cp >> 8];
  const uint32_t v = (l2[blk * 128u + ((cp & 255u) >> 1)] >> ((cp & 1u) * 4u)) & 15u;
  // table values: 0 other, 1 Lu|Lt, 2 Ll, 3 Lm|Lo, 4 M, 5 N, 6 \s
  return v;
}

// Whether a position whose left character has class x (code point cx) and
// whose right character has class y (code point cy) is a synchronizing
// boundary of the o200k-style pattern: every text with these two characters
// there has a piece boundary between them, the pieces to the right depend on
// the left only through x, and the pieces to the left depend on the right
// only through y.  From the alternatives:
//   - a number run head always starts a piece (no set before it takes digits);
//   - a letter is safe after a number or CR/LF (neither can be a prefix), and
//     an upper-case letter after a lower-case one (a lower-case character is
//     only ever matched by the lower-case part of a piece, which ends at the
//     next upper-case letter);
//   - whitespace other than CR/LF is safe after letters, marks, numbers and
//     symbols (no set before it takes it, and it only begins pieces);
//   - CR/LF is safe after letters and numbers (after a symbol or a mark it
//     can be absorbed by a symbol piece);
//   - a symbol is safe after a letter unless it is an apostrophe (a
//     contraction suffix), after a number, after CR/LF unless it is "/" (a
//     symbol piece absorbs CR/LF and "/" after it), and after whitespace other
//     than U+0020 (which would join it);
//   - marks are never safe: they can extend a letter run and a symbol run.
__host__ __device__ constexpr bool o2_sync(uint32_t x, uint32_t y, uint32_t cx, uint32_t cy) {
  switch (y) {
    case O2_N: return x != O2_N && x != O2_NONE;
    case O2_UP: return x == O2_N || x == O2_NL || x == O2_LO;
    case O2_LO:
    case O2_BO: return x == O2_N || x == O2_NL;
    case O2_WS: return o2_letter(x) || x == O2_MK || x == O2_N || x == O2_O;
    case O2_NL: return o2_letter(x) || x == O2_N;
    case O2_O:
      return (o2_letter(x) && cy != 0x27u) || x == O2_N || (x == O2_NL && cy != 0x2Fu) ||
             (x == O2_WS && cx != 0x20u);
    default: return false;
  }
}

// Byte length of the UTF-8 sequence a lead byte starts (1 for bytes that
// cannot lead: such text is invalid and its output is discarded).
__host__ __device__ inline uint32_t o2_lead_len(uint32_t b) {
  return b < 0xC0u ? 1u : b < 0xE0u ? 2u : b < 0xF0u ? 3u : b < 0xF8u ? 4u : 1u;
}

// The request as seen from one tile: window bytes and codes in LDS, the rest
// in global memory.  Positions are window indices (the window starts at text
// position w0); they may lie outside the window.
typedef __attribute__((address_space(3))) const uint8_t lds_u8;    // a byte in LDS
typedef __attribute__((address_space(3))) const uint32_t lds_u32;  // a word in LDS
typedef __attribute__((address_space(3))) const int32_t lds_i32;   // a signed word in LDS

// Class-set bitmaps of a tile's window: bit q of bitmap k (word q / 32 of
// its PT_WIN / 32 words) tells whether window index q belongs to set k.  In a
// "run" set the continuation bytes of the text are members too, so that a run
// scan can step byte by byte.  In a "last" set only the characters of the
// set are members (their first bytes): such a set finds the last character of
// a class inside a run.  Document starts and positions outside the text are
// in no set (a run stops there).
constexpr int WALK_BITMAPS = 9;
constexpr int WB_DIGITS = 8;  // both patterns: ASCII digits (a run of them is cut in threes from its head)
constexpr int WIN_WORDS = PT_WIN / 32;

// First window index p >= q (0 <= q < PT_WIN) whose bit in bitmap b is 0, or
// PT_WIN when every bit from q to the window end is 1.
__device__ __forceinline__ int64_t win_next_zero(lds_u32* b, int64_t q) {
  uint32_t wi = (uint32_t)q >> 5;
  uint32_t x = ~b[wi] & (0xFFFFFFFFu << ((uint32_t)q & 31u));
  while (x == 0u) {
    if (++wi >= (uint32_t)WIN_WORDS) return PT_WIN;
    x = ~b[wi];
  }
  return (int64_t)(wi * 32u + (uint32_t)__builtin_ctz(x));
}

// Last window index in [a, e) whose bit in bitmap b is 1, or -1
// (0 <= a, e <= PT_WIN).
__device__ __forceinline__ int64_t win_last_one(lds_u32* b, int64_t a, int64_t e) {
  if (e <= a) return -1;
  const int32_t wa = (int32_t)(a >> 5);
  int32_t wi = (int32_t)((e - 1) >> 5);
  uint32_t x = b[wi] & (0xFFFFFFFFu >> (31u - ((uint32_t)(e - 1) & 31u)));
  for (;;) {
    if (wi == wa) x &= 0xFFFFFFFFu << ((uint32_t)a & 31u);
    if (x) return (int64_t)wi * 32 + 31 - __builtin_clz(x);
    if (--wi < wa) return -1;
    x = b[wi];
  }
}

// Position of the set bit of rank r (counted from bit 0) of m; r < popcount(m).
__host__ __device__ inline uint32_t select_bit64(uint64_t m, uint32_t r) {
  uint32_t p = 0;
  uint32_t x = (uint32_t)m;
  uint32_t c = (uint32_t)__builtin_popcount(x);
  if (r >= c) {
    r -= c;
    p = 32;
    x = (uint32_t)(m >> 32);
  }
#pragma unroll
  for (int w = 16; w >= 1; w >>= 1) {
    c = (uint32_t)__builtin_popcount(x & ((1u << w) - 1u));
    if (r >= c) {
      r -= c;
      p += (uint32_t)w;
      x >>= w;
    }
  }
  return p;
}

// The o200k-style bitmaps: runs of [Lu Lt Lm Lo M], of [Ll Lm Lo M], of
// [^\s\p{L}\p{N}] and of \s; the last Lm/Lo letter or mark, and the last CR/LF.
enum : int { O2B_UB = 0, O2B_LB = 1, O2B_OS = 2, O2B_SP = 3, O2B_BM = 4, O2B_NL = 5 };
constexpr uint32_t O2B_RUNS = (1u << O2B_UB) | (1u << O2B_LB) | (1u << O2B_OS) | (1u << O2B_SP);
__host__ __device__ constexpr uint32_t o2_bits_of(uint32_t c) {
  uint32_t m = 0;
  if (c == O2_UP || c == O2_BO || c == O2_MK) m |= 1u << O2B_UB;
  if (c == O2_LO || c == O2_BO || c == O2_MK) m |= 1u << O2B_LB;
  if (c == O2_O || c == O2_MK) m |= 1u << O2B_OS;
  if (c == O2_WS || c == O2_NL) m |= 1u << O2B_SP;
  if (c == O2_BO || c == O2_MK) m |= 1u << O2B_BM;
  if (c == O2_NL) m |= 1u << O2B_NL;
  return m;
}

// Branch-free forms of o2_sync and o2_bits_of for the tile kernel (a switch
// over classes becomes a tree of divergent branches on the GPU), as bit tables
// built from the functions themselves.  o2_sync depends on the two code
// points only through "cy is an apostrophe", "cy is a slash" and "cx is
// U+0020": one 64-bit table per case, bit 8y + x.
constexpr uint64_t o2_sync_table(uint32_t cx, uint32_t cy) {
  uint64_t t = 0;
  for (uint32_t y = 0; y < 8; ++y)
    for (uint32_t x = 0; x < 8; ++x)
      if (o2_sync(x, y, cx, cy)) t |= 1ull << (8 * y + x);
  return t;
}
__device__ __forceinline__ bool o2_sync_bits(uint32_t x, uint32_t y, uint32_t cx, uint32_t cy) {
  constexpr uint64_t T0 = o2_sync_table(0x80, 0x80), T1 = o2_sync_table(0x80, 0x27), T2 = o2_sync_table(0x80, 0x2F);
  constexpr uint64_t T3 = o2_sync_table(0x20, 0x80), T4 = o2_sync_table(0x20, 0x27), T5 = o2_sync_table(0x20, 0x2F);
  const bool sp = cx == 0x20u;
  const uint64_t t = cy == 0x27u ? (sp ? T4 : T1) : cy == 0x2Fu ? (sp ? T5 : T2) : (sp ? T3 : T0);
  return x < 8u && y < 8u && ((t >> (8u * y + x)) & 1u) != 0u;
}
// The classes (bit c) whose characters are in bitmap k, continuation bytes
// (class O2_NONE) in every run set.
constexpr uint32_t o2_bitmap_classes(int k) {
  uint32_t m = ((O2B_RUNS >> k) & 1u) << O2_NONE;
  for (uint32_t c = 0; c < 15; ++c)
    if ((o2_bits_of(c) >> k) & 1u) m |= 1u << c;
  return m;
}

// The runs through the window's end (far_serve): per run bitmap, where its
// run through the window's end ends and the last tracked character past the
// window (-1 if none), both window indices, and their state (FAR_NONE, then
// FAR_BUSY while a wave finds them, FAR_READY once they hold their values).
enum : uint32_t { FAR_NONE = 0, FAR_BUSY = 1, FAR_READY = 2 };
struct FarRuns {
  int32_t end[WALK_BITMAPS], last[WALK_BITMAPS];
  uint32_t state[WALK_BITMAPS];
};
typedef __attribute__((address_space(3))) FarRuns lds_far;

struct O2View {
  lds_u8* buf;          // window bytes at PT_PAD + q, q in [-PT_PAD, PT_WIN + 16)
  lds_u8* code;         // window codes at PT_PAD + q: class | CODE_DOCSTART
  lds_u8* l1;           // class table levels
  lds_u8* l2;
  const uint8_t* text;  // the request
  int64_t w0, n;
  int64_t doc_after;    // first document start at or after w0 + PT_WIN (n if none)
  lds_u32* bits;        // the window's class-set bitmaps, WIN_WORDS words each
  lds_u8* asc;          // the pattern's class of every ASCII character
  lds_far* far;         // the runs through the window's end (see far_serve)

  __device__ bool in_win(int64_t q) const { return q >= 0 && q < PT_WIN; }
  __device__ uint32_t byte(int64_t q) const {
    return (q >= -PT_PAD && q < PT_WIN + 16) ? (uint32_t)buf[PT_PAD + q] : (uint32_t)text[w0 + q];
  }
  // q is past the end of the document of a piece that starts before q
  __device__ bool past(int64_t q) const {
    if (w0 + q >= n) return true;
    if (in_win(q)) return (code[PT_PAD + q] & 0x80u) != 0u;
    return q >= PT_WIN && w0 + q >= doc_after;
  }
  __device__ uint32_t clen(int64_t q) const { return o2_lead_len(byte(q)); }
  __device__ uint32_t cls(int64_t q) const {
    if (in_win(q)) return code[PT_PAD + q] & 15u;
    const uint32_t b0 = byte(q);
    if (b0 < 0x80u) return o2_table_class(l1, l2, b0);
    const uint32_t L = o2_lead_len(b0);
    if (L == 1u) return O2_NONE;
    uint32_t cp = b0 & (0x7Fu >> L);
    for (uint32_t k = 1; k < L; ++k) {
      if (w0 + q + k >= n) return O2_NONE;
      cp = (cp << 6) | (byte(q + k) & 0x3Fu);
    }
    return cp < 0x110000u ? o2_table_class(l1, l2, cp) : O2_NONE;
  }
};

// Class of a character outside the window (rare: walks that run past it).
__device__ __noinline__ uint32_t o2_cls_far(const O2View v, int64_t q) { return v.cls(q); }

// Class-set masks (bit c set when class c is in the set).
constexpr uint32_t M_UB = (1u << O2_UP) | (1u << O2_BO) | (1u << O2_MK);   // [\p{Lu}\p{Lt}\p{Lm}\p{Lo}\p{M}]
constexpr uint32_t M_LB = (1u << O2_LO) | (1u << O2_BO) | (1u << O2_MK);   // [\p{Ll}\p{Lm}\p{Lo}\p{M}]
constexpr uint32_t M_BM = (1u << O2_BO) | (1u << O2_MK);                   // in both letter sets
constexpr uint32_t M_OS = (1u << O2_O) | (1u << O2_MK);                    // [^\s\p{L}\p{N}]
constexpr uint32_t M_SP = (1u << O2_WS) | (1u << O2_NL);                   // \s
constexpr uint32_t M_PF = (1u << O2_O) | (1u << O2_MK) | (1u << O2_WS);    // [^\r\n\p{L}\p{N}]

// The class set of run bitmap k (0 for a bitmap that is not a run set), and
// the classes whose last character the scans of that set track.
__host__ __device__ inline uint32_t o2_run_mask(int k) {
  return k == O2B_UB ? M_UB : k == O2B_LB ? M_LB : k == O2B_OS ? M_OS : k == O2B_SP ? M_SP : 0u;
}
__host__ __device__ inline uint32_t o2_run_track(int k) { return k == O2B_UB ? M_BM : k == O2B_SP ? 1u << O2_NL : 0u; }

// The part of a run scan past the window (rare): from q (a character start
// past the window), while the class is in `mask`; `last` becomes the start of
// the last character whose class is in `track`.  The text is read 16 bytes a
// step (all loads of a step in flight together), and the characters that lie
// whole in those bytes are decoded and classed from registers (ASCII from the
// ASCII table, others from the class table with tcls), so that a run of tens
// of thousands of characters costs thousands of load round trips, not tens of
// thousands.
struct ScanEnd {
  int64_t q, last;
};
template <class TClsF>
__device__ __forceinline__ ScanEnd scan_far(const O2View& v, int64_t q, uint32_t mask, uint32_t track, int64_t last,
                                            TClsF tcls) {
  const int64_t lim = (v.doc_after < v.n ? v.doc_after : v.n) - v.w0;  // where the document ends
#pragma unroll 1
  while (q < lim) {
    const uint8_t* src = v.text + (v.w0 + q);
    const int64_t avail = lim - q;  // bytes before the end (> 0)
    uint32_t B[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) B[i] = i < avail ? (uint32_t)src[i] : 0u;
    uint32_t o = 0;      // start of the next character in the step's bytes
    bool stop = false;   // a character did not fit, or the run ended
    bool end = false;    // the run ended at o
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (!stop && (uint32_t)i == o) {
        const uint32_t b0 = B[i];
        const uint32_t L = o2_lead_len(b0);  // (1 for bytes that cannot lead)
        if ((int64_t)i + (int64_t)L > (avail < 16 ? avail : 16)) {
          stop = true;  // not whole in this step: the next step starts with it
        } else {
          uint32_t c;
          if (b0 < 0x80u) {
            c = v.asc[b0];
          } else if (L == 1u) {
            c = O2_NONE;  // a stray continuation byte: invalid text
          } else {
            uint32_t cp = b0 & (0x7Fu >> L);
#pragma unroll
            for (int k = 1; k < 4; ++k)
              if ((uint32_t)k < L && i + k < 16) cp = (cp << 6) | (B[i + k] & 0x3Fu);
            c = cp < 0x110000u ? tcls(cp) : O2_NONE;
          }
          if (!((mask >> c) & 1u)) {
            stop = true;
            end = true;
          } else {
            if ((track >> c) & 1u) last = q + i;
            o = (uint32_t)i + L;
          }
        }
      }
    }
    q += o;
    if (end || o == 0u) break;  // (o == 0: a character cut by the end of the text)
  }
  return {q, last};
}

// Where the runs that hold the window's last character end past the window.
// Every walk's scan that reaches the window's end continues the same run past
// it: from the end of the window's last character, while the class is in the
// run set.  So a tile finds that continuation once per run set, when a walk
// first needs it, on one wave: first over the 16 bytes staged past the window
// (one lane), then, for a run that goes on beyond them, over the text with
// the whole wave, 16 bytes per lane per step (far_run_wave).
struct FarRun {
  int64_t end, last;
  bool open;  // the run goes on past the staged bytes
};
template <class TClsF>
__device__ __forceinline__ FarRun far_run_staged(const O2View& v, int64_t q, int64_t lim, uint32_t mask, uint32_t track,
                                                 TClsF tcls) {
  int64_t last = -1;
#pragma unroll 1
  for (;;) {
    if (q >= lim) return {q, last, false};          // the document ends
    if (q + 4 > PT_WIN + 16) return {q, last, true};  // (the next character may not be staged whole)
    const uint32_t b0 = v.buf[PT_PAD + q];
    const uint32_t L = o2_lead_len(b0);
    if (q + (int64_t)L > lim) return {q, last, false};  // cut by the end: not in any set
    uint32_t c;
    if (b0 < 0x80u) {
      c = v.asc[b0];
    } else if (L == 1u) {
      c = O2_NONE;
    } else {
      uint32_t cp = b0 & (0x7Fu >> L);
      for (uint32_t k = 1; k < L; ++k) cp = (cp << 6) | (v.buf[PT_PAD + q + k] & 0x3Fu);
      c = cp < 0x110000u ? tcls(cp) : O2_NONE;
    }
    if (!((mask >> c) & 1u)) return {q, last, false};
    if ((track >> c) & 1u) last = q;
    q += L;
  }
}

// The same past the staged bytes, on one wave: lane i takes the characters
// that start in [pos + 16i, pos + 16i + 16), decoded from 19 bytes in
// registers; the first lane that finds the run's end gives it, and the last
// tracked character is the latest one before that end.  Every lane of the
// wave calls it with the same arguments.
template <class TClsF>
__device__ __forceinline__ FarRun far_run_wave(const O2View& v, int64_t pos, int64_t last, int64_t lim, uint32_t mask,
                                               uint32_t track, TClsF tcls) {
  const uint32_t lane = threadIdx.x & 63u;
  constexpr uint32_t NONE = 0xFFFFFFFFu;
#pragma unroll 1
  for (;;) {
    const int64_t a = pos + 16 * (int64_t)lane;
    const int64_t avail = lim - a;  // bytes of the lane's reach before the end (may be <= 0)
    uint32_t B[19];
#pragma unroll
    for (int i = 0; i < 19; ++i) B[i] = i < avail ? (uint32_t)v.text[v.w0 + a + i] : 0u;
    // a character that starts before a belongs to the lane before
    uint32_t o = (B[0] & 0xC0u) == 0x80u ? ((B[1] & 0xC0u) == 0x80u ? ((B[2] & 0xC0u) == 0x80u ? 3u : 2u) : 1u) : 0u;
    uint32_t stop = NONE;    // offset of the run's end in the lane's part
    uint32_t mylast = NONE;  // offset of the lane's last tracked character
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      if (stop == NONE && (uint32_t)i == o) {
        if ((int64_t)i >= avail) {
          stop = (uint32_t)i;  // the document ends
        } else {
          const uint32_t b0 = B[i];
          const uint32_t L = o2_lead_len(b0);
          uint32_t c;
          if ((int64_t)i + (int64_t)L > avail) {
            c = O2_NONE;  // cut by the end
          } else if (b0 < 0x80u) {
            c = v.asc[b0];
          } else if (L == 1u) {
            c = O2_NONE;
          } else {
            uint32_t cp = b0 & (0x7Fu >> L);
#pragma unroll
            for (int k = 1; k < 4; ++k)
              if ((uint32_t)k < L) cp = (cp << 6) | (B[i + k] & 0x3Fu);
            c = cp < 0x110000u ? tcls(cp) : O2_NONE;
          }
          if (!((mask >> c) & 1u)) {
            stop = (uint32_t)i;
          } else {
            if ((track >> c) & 1u) mylast = (uint32_t)i;
            o = (uint32_t)i + L;
          }
        }
      }
    }
    const uint64_t ends = __ballot(stop != NONE);
    const uint32_t first = ends ? (uint32_t)__builtin_ctzll(ends) : 64u;  // lane with the run's end
    // latest tracked character in the lanes up to that one (offsets from pos, + 1; 0 for none)
    uint32_t t = (lane <= first && mylast != NONE) ? 16u * lane + mylast + 1u : 0u;
#pragma unroll
    for (int d = 1; d < 64; d <<= 1) {
      const uint32_t u = (uint32_t)__shfl_xor((int)t, d, 64);
      t = u > t ? u : t;
    }
    if (t != 0u) last = pos + (int64_t)(t - 1u);
    if (ends) {
      const uint32_t st = (uint32_t)__builtin_amdgcn_readlane((int)stop, (int)first);
      return {pos + 16 * (int64_t)first + st, last, false};
    }
    pos += 16 * 64;
  }
}

// Finds, on one wave, the runs through the window's end of the run bitmaps
// in `sets` (bit k: bitmap k) that are not found yet: lane 0 takes the staged
// bytes, then the whole wave reads on if the run goes further.  A set that
// another wave is finding is waited for (that wave waits for nothing).  The
// walks ask for a set only when a scan of theirs reaches the window's end
// (FullView), so most tiles find none.  mask_of / track_of give a bitmap's
// class set and tracked classes, tcls the class of a non-ASCII code point.
// Every lane of the wave calls it with the same `sets`.
template <class MaskF, class TrackF, class TClsF>
__device__ __forceinline__ void far_serve(const O2View& v, uint32_t sets, MaskF mask_of, TrackF track_of, TClsF tcls) {
  const uint32_t lane = threadIdx.x & 63u;
  const int64_t lim = (v.doc_after < v.n ? v.doc_after : v.n) - v.w0;  // where the document ends
  uint32_t* state = (uint32_t*)v.far->state;
#pragma unroll 1
  for (int k = 0; k < WALK_BITMAPS; ++k) {
    if (!((sets >> k) & 1u)) continue;
    uint32_t mine = 0;
    if (lane == 0u) mine = atomicCAS(&state[k], FAR_NONE, FAR_BUSY) == FAR_NONE;
    mine = (uint32_t)__builtin_amdgcn_readfirstlane((int)mine);
    if (!mine) {
      while (__hip_atomic_load(&state[k], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) != FAR_READY)
        __builtin_amdgcn_s_sleep(1);
      continue;
    }
    const uint32_t mk = mask_of(k), tk = track_of(k);
    int32_t fe = 0, fl = -1, fo = 0;
    if (lane == 0u) {
      int r0 = PT_WIN - 1;  // the window's last character
      while (r0 > PT_WIN - 4 && (v.buf[PT_PAD + r0] & 0xC0u) == 0x80u) --r0;
      const uint32_t c_last = v.code[PT_PAD + r0] & 15u;
      const int64_t start = r0 + (int64_t)o2_lead_len(v.buf[PT_PAD + r0]);
      FarRun f{start, -1, false};
      if (mk != 0u && ((mk >> c_last) & 1u)) f = far_run_staged(v, start, lim, mk, tk, tcls);
      fe = (int32_t)f.end;
      fl = (int32_t)f.last;
      fo = f.open;
    }
    fe = __builtin_amdgcn_readfirstlane(fe);
    fl = __builtin_amdgcn_readfirstlane(fl);
    if (__builtin_amdgcn_readfirstlane(fo)) {
      const FarRun f = far_run_wave(v, fe, fl, lim, mk, tk, tcls);
      fe = (int32_t)f.end;
      fl = (int32_t)f.last;
    }
    if (lane == 0u) {
      v.far->end[k] = fe;
      v.far->last[k] = fl;
      __hip_atomic_store(&state[k], FAR_READY, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    }
  }
}

// far_serve for the o200k-style pattern, out of line (rare, and its
// registers would otherwise weigh on the whole kernel).
__device__ __noinline__ void o2_far_serve(const O2View v, uint32_t sets) {
  far_serve(v, sets, o2_run_mask, o2_run_track, [&](uint32_t cp) { return o2_table_class(v.l1, v.l2, cp); });
}

__device__ __noinline__ ScanEnd o2_scan_far(const O2View v, int64_t q, uint32_t mask, uint32_t track, int64_t last) {
  return scan_far(v, q, mask, track, last, [&](uint32_t cp) { return o2_table_class(v.l1, v.l2, cp); });
}

// Two ways to read a walk's positions (P is the position type).  The piece
// rules below take either.
//
// WinView: the window in LDS only, with 32-bit positions and no branch to
// global memory; every position at or past the window's end reads as past
// the text.  Its answer is the piece's end when no run scan reached the
// window's end (`out`) and the end lies at least WIN_MARGIN bytes before it:
// a rule reads at most WIN_MARGIN - 1 bytes past the end it returns.  Else
// the piece is taken again with the full view.
constexpr int WIN_MARGIN = 5;
struct WinView {
  lds_u8* buf;
  lds_u8* code;
  lds_u32* bits;
  int32_t qn;        // window index of the text end, at most PT_WIN
  bool out = false;  // a run scan reached the window's end

  __device__ uint32_t byte(int32_t q) const { return buf[PT_PAD + q]; }
  __device__ uint32_t clen(int32_t q) const { return o2_lead_len(byte(q)); }
  __device__ uint32_t cls(int32_t q) const { return code[PT_PAD + q] & 15u; }
  __device__ bool past(int32_t q) const { return q >= qn || (code[PT_PAD + q] & 0x80u) != 0u; }
  // advance from q (> the piece start, a character start) while the class
  // is in run bitmap rb; `last` receives the start of the last character
  // in bitmap tb (-1 for none), or keeps its value
  __device__ int32_t scan(int32_t q, uint32_t, uint32_t, int32_t& last, int rb, int tb) {
    if (q >= PT_WIN) {
      out = true;
      return q;
    }
    const int32_t p = (int32_t)win_next_zero(bits + rb * WIN_WORDS, q);
    if (tb >= 0) {
      const int32_t t = (int32_t)win_last_one(bits + tb * WIN_WORDS, q, p);
      if (t >= 0) last = t;
    }
    out = out || p >= PT_WIN;
    return p;
  }
};

// FullView: any position of the request (outside the window from the text
// and the class table, through the out-of-line helpers of the pattern).
template <uint32_t (*FAR_CLS)(const O2View, int64_t), ScanEnd (*FAR_SCAN)(const O2View, int64_t, uint32_t, uint32_t, int64_t)>
struct FullView {
  const O2View& v;
  int need = -1;  // a run bitmap whose run through the window's end is not found yet (see scan)
  __device__ uint32_t byte(int64_t q) const { return v.byte(q); }
  __device__ uint32_t clen(int64_t q) const { return v.clen(q); }
  __device__ uint32_t cls(int64_t q) const { return v.in_win(q) ? (uint32_t)(v.code[PT_PAD + q] & 15u) : FAR_CLS(v, q); }
  __device__ bool past(int64_t q) const { return need >= 0 || v.past(q); }
  // as WinView::scan, with `mask` the classes of the run for the part past
  // the window.  A run that holds the window's last character ends where the
  // tile's run of that bitmap through the window's end ends (far_serve); when
  // that is not found yet, the scan sets `need`, and from then on every scan
  // returns at once and every position reads as past the text (the piece's
  // end is then of no use: the walk asks for the run and takes the piece
  // again).
  __device__ int64_t scan(int64_t q, uint32_t mask, uint32_t track, int64_t& last, int rb, int tb) {
    if (need >= 0) return q;
    if (q < PT_WIN) {
      const int64_t p = win_next_zero(v.bits + rb * WIN_WORDS, q);
      if (tb >= 0) {
        const int64_t t = win_last_one(v.bits + tb * WIN_WORDS, q, p);
        if (t >= 0) last = t;
      }
      if (p < PT_WIN) return p;
      if (__hip_atomic_load((const uint32_t*)&v.far->state[rb], __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) != FAR_READY) {
        need = rb;
        return PT_WIN;
      }
      if (tb >= 0 && v.far->last[rb] >= 0) last = v.far->last[rb];
      return v.far->end[rb];
    }
    const ScanEnd f = FAR_SCAN(v, q, mask, track, last);
    last = f.last;
    return f.q;
  }
};

// End (window index) of the piece that starts at s, by the pattern's
// alternatives in order.  Always > s.  Every alternative is evaluated with
// two run scans ("advance while the character's class is in a set"): the
// upper-case letter body after the first character, then the run the chosen
// alternative ends with; the first alternative that matches is taken.
template <class V, class P>
__device__ __forceinline__ P o2_end(V& v, const P s) {
  auto stop = [&](P q) { return q > s && v.past(q); };
  const uint32_t c0 = v.cls(s);
  const P s1 = s + (P)v.clen(s);
  const bool pfx = ((M_PF >> c0) & 1u) != 0u && !stop(s1);
  const bool ub0 = ((M_UB >> c0) & 1u) != 0u;
  // the letter bodies after the prefix (a) and from s (b), both runs of the
  // upper-case set from s1 (a character at s in that set cannot be a prefix
  // but a mark, which is both): where each ends and its last "both"
  // character
  P qu = s1, lu = -1;
  if (pfx || ub0) qu = v.scan(s1, M_UB, M_BM, lu, O2B_UB, O2B_BM);
  const P qa = qu, lba = lu;
  const P qb = ub0 ? qu : s;
  const P lbb = lu >= 0 ? (ub0 ? lu : (P)-1) : ((M_BM >> c0) & 1u) ? s : (P)-1;
  const bool loa = pfx && !stop(qa) && v.cls(qa) == O2_LO;
  const bool lob = !stop(qb) && v.cls(qb) == O2_LO;
  // P1 with the prefix, P1 without, P2 with, P2 without: where the
  // lower-case set starts (in the first two cases the character at `from`
  // is in that set; in the last two, P2 with an empty lower-case part, it
  // is not)
  P from = -1;
  bool from_in = true;
  if (pfx && (loa || lba >= 0)) from = loa ? qa : lba;
  else if (lob || lbb >= 0) from = lob ? qb : lbb;
  else if (pfx && qa > s1) from = qa, from_in = false;
  else if (qb > s) from = qb, from_in = false;
  // P3: one to three numbers
  if (from < 0 && c0 == O2_N) {
    P q = s1;
    for (int k = 1; k < 3 && !stop(q) && v.cls(q) == O2_N; ++k) q += (P)v.clen(q);
    return q;
  }
  // the closing run: the lower-case set (P1, P2); symbols and marks after an
  // optional U+0020 (P4); whitespace, with its last CR/LF (P5-P7)
  int alt;
  P q0, last = -1;
  uint32_t mask, track = 0u;
  int rb, tb = -1;
  if (from >= 0) {
    alt = 1;  // (from > s unless the character at s is in the lower-case set)
    q0 = from_in ? from + (P)v.clen(from) : from;
    mask = M_LB;
    rb = O2B_LB;
  } else {
    const P st = (v.byte(s) == 0x20u && !stop(s1) && ((M_OS >> v.cls(s1)) & 1u)) ? s1 : s;
    if ((M_OS >> v.cls(st)) & 1u) {
      alt = 4;
      q0 = st + (P)v.clen(st);
      mask = M_OS;
      rb = O2B_OS;
    } else if ((M_SP >> c0) & 1u) {
      alt = 5;
      q0 = s1;
      mask = M_SP;
      track = 1u << O2_NL;
      rb = O2B_SP;
      tb = O2B_NL;
      if (c0 == O2_NL) last = s;
    } else {
      return s1;  // only invalid text gets here
    }
  }
  const P e = v.scan(q0, mask, track, last, rb, tb);
  if (alt == 1) {
    // the optional case-insensitive contraction
    if (stop(e) || v.byte(e) != 0x27u || stop(e + 1)) return e;
    const uint32_t b1 = v.byte(e + 1);
    if (b1 == 0xC5u && !stop(e + 2) && v.byte(e + 2) == 0xBFu) return e + 3;  // U+017F folds to s
    const uint32_t f1 = b1 | 0x20u;
    if (f1 == 's' || f1 == 't' || f1 == 'm' || f1 == 'd') return e + 2;
    if ((f1 == 'r' || f1 == 'v' || f1 == 'l') && !stop(e + 2)) {
      const uint32_t f2 = v.byte(e + 2) | 0x20u;
      if ((f1 == 'l' && f2 == 'l') || (f1 != 'l' && f2 == 'e')) return e + 3;
    }
    return e;
  }
  if (alt == 4) {  // then CR/LF and "/"
    P q = e;
    while (!stop(q) && (v.byte(q) == 0x0Au || v.byte(q) == 0x0Du || v.byte(q) == 0x2Fu)) ++q;
    return q;
  }
  if (last >= 0) return last + 1;  // \s*[\r\n]+
  if (stop(e)) return e;           // \s+(?!\S) at the end of the text
  // \s+(?!\S) gives back the last character, if there are two or more
  for (P r = e - 1; r > s && r >= e - 4; --r)
    if ((v.byte(r) & 0xC0u) != 0x80u) return r;
  return e;  // else \s+
}

// The piece's end with the full view (rare: pieces at the window's end), or
// -1 - k when the run through the window's end of bitmap k is needed first.
__device__ __noinline__ int64_t o2_end_full(const O2View v, int64_t s) {
  FullView<o2_cls_far, o2_scan_far> f{v};
  const int64_t e = o2_end(f, s);
  return f.need >= 0 ? -1 - (int64_t)f.need : e;
}

// End (window index) of the piece that starts at s (0 <= s < PT_WIN), or
// -1 - k as o2_end_full.
__device__ __forceinline__ int64_t o2_piece_end(const O2View& v, int64_t s) {
  WinView f{v.buf, v.code, v.bits, (int32_t)(v.n - v.w0 < PT_WIN ? v.n - v.w0 : PT_WIN)};
  const int32_t e = o2_end(f, (int32_t)s);
  if (!f.out && e + WIN_MARGIN <= PT_WIN) return e;
  return o2_end_full(v, s);
}

}  // namespace tt
