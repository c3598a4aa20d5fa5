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

__host__ __device__ inline bool o2_letter(uint32_t c) { return c == O2_UP || c == O2_LO || c == O2_BO; }
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
__host__ __device__ inline bool o2_sync(uint32_t x, uint32_t y, uint32_t cx, uint32_t cy) {
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
typedef __attribute__((address_space(3))) const uint8_t lds_u8;  // a byte in LDS

struct O2View {
  lds_u8* buf;          // window bytes at PT_PAD + q, q in [-PT_PAD, PT_WIN + 16)
  lds_u8* code;         // window codes at PT_PAD + q: class | CODE_DOCSTART
  lds_u8* l1;           // class table levels
  lds_u8* l2;
  const uint8_t* text;  // the request
  int64_t w0, n;
  int64_t doc_after;    // first document start at or after w0 + PT_WIN (n if none)

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

// End (window index) of the piece that starts at s, by the pattern's
// alternatives in order.  Always > s.  Every alternative is evaluated with the
// same few scans ("advance while the character's class is in a set"), and the
// first one that matches is taken: the lanes of a wave, each on its own
// piece, then run the same instructions.
__device__ __forceinline__ int64_t o2_piece_end(const O2View& v, int64_t s) {
  auto stop = [&](int64_t q) { return q > s && v.past(q); };
  auto cls = [&](int64_t q) -> uint32_t { return v.in_win(q) ? (uint32_t)(v.code[PT_PAD + q] & 15u) : o2_cls_far(v, q); };
  // advance from q while the class is in `mask`; `last` receives the start
  // of the last character whose class is in `track` (or keeps its value)
  auto scan = [&](int64_t q, uint32_t mask, uint32_t track, int64_t& last) -> int64_t {
    for (;;) {
      if (stop(q)) return q;
      const uint32_t c = cls(q);
      if (!((mask >> c) & 1u)) return q;
      if ((track >> c) & 1u) last = q;
      q += v.clen(q);
    }
  };
  const uint32_t c0 = cls(s);
  const int64_t l0 = v.clen(s);
  const bool pfx = ((M_PF >> c0) & 1u) != 0u && !stop(s + l0);
  int64_t unused = -1;
  // the letter bodies after the prefix (a) and from s (b): the run of the
  // upper-case set, its last "both" character, and the class after it
  const int64_t ba = s + l0;
  int64_t lba = -1, lbb = -1;
  const int64_t qa = pfx ? scan(ba, M_UB, M_BM, lba) : ba;
  const int64_t qb = scan(s, M_UB, M_BM, lbb);
  const bool loa = pfx && !stop(qa) && cls(qa) == O2_LO;
  const bool lob = !stop(qb) && cls(qb) == O2_LO;
  // P1 with the prefix, P1 without, P2 with, P2 without: where the
  // lower-case set starts
  int64_t from = -1;
  if (pfx && (loa || lba >= 0)) from = loa ? qa : lba;
  else if (lob || lbb >= 0) from = lob ? qb : lbb;
  else if (pfx && qa > ba) from = qa;
  else if (qb > s) from = qb;
  if (from >= 0) {
    const int64_t e = scan(from, M_LB, 0u, unused);
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
  // P3: one to three numbers
  if (c0 == O2_N) {
    int64_t q = s + l0;
    for (int k = 1; k < 3 && !stop(q) && cls(q) == O2_N; ++k) q += v.clen(q);
    return q;
  }
  // P4: optional U+0020, symbols and marks, then CR/LF and "/"
  const int64_t st = (v.byte(s) == 0x20u && !stop(s + 1) && ((M_OS >> cls(s + 1)) & 1u)) ? s + 1 : s;
  if ((M_OS >> cls(st)) & 1u) {
    int64_t q = scan(st, M_OS, 0u, unused);
    while (!stop(q) && (v.byte(q) == 0x0Au || v.byte(q) == 0x0Du || v.byte(q) == 0x2Fu)) ++q;
    return q;
  }
  // P5-P7: whitespace
  if ((M_SP >> c0) & 1u) {
    int64_t last_nl = -1, last_start = s;
    const int64_t q = scan(s, M_SP, 1u << O2_NL, last_nl);
    if (last_nl >= 0) return last_nl + 1;  // \s*[\r\n]+
    if (stop(q)) return q;                  // \s+(?!\S) at the end of the text
    // \s+(?!\S) gives back the last character, if there are two or more
    for (int64_t r = q - 1; r > s && r >= q - 4; --r)
      if ((v.byte(r) & 0xC0u) != 0x80u) {
        last_start = r;
        break;
      }
    return last_start > s ? last_start : q;  // else \s+
  }
  return s + l0;  // only invalid text gets here
}

}  // namespace tt
