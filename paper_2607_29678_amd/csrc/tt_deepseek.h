// The DeepSeek-style pattern (Sec. 4.1: DeepSeek-family tokenizers apply three
// splitters in sequence; their composition folds into one per-character
// predicate when each splitter re-splits every piece of the stage before and
// unmatched stretches survive as pieces).  The splitters, in order:
//   S1  \p{N}{1,3}
//   S2  runs of CJK ideographs U+4E00-9FA5, hiragana U+3040-309F, katakana U+30A0-30FF
//   S3  D1 [ASCII punctuation or symbol][A-Za-z]+
//       D2 [^\r\n\p{L}\p{P}\p{S}]?[\p{L}\p{M}]+
//       D3 U+0020? [\p{P}\p{S}]+ [\r\n]*
//       D4 \s*[\r\n]+    D5 \s+(?!\S)    D6 \s+
//
// A stretch of numbers, a stretch of the CJK/kana set and a stretch of
// everything else ("groups") are pieces of the first two stages, so every
// group change is a piece boundary that no context moves, and the third
// splitter runs inside one group stretch at a time, which it sees as the
// whole text.  The tile kernel walks the pieces between synchronizing
// positions as for the o200k-style pattern (tt_o200k.h), with the walk of a
// piece bounded by its group stretch.
#pragma once

#include "tt_internal.h"
#include "tt_o200k.h"

namespace tt {

// Classes of the DeepSeek-style pattern (4 bits of a window code), as in the
// generated table.
enum : uint32_t {
  DS_O = 0,    // none of the others (controls, format characters, unassigned)
  DS_AL = 1,   // ASCII letter
  DS_L = 2,    // other letter
  DS_M = 3,    // mark
  DS_N = 4,    // \p{N}
  DS_AP = 5,   // ASCII punctuation or symbol
  DS_PS = 6,   // other punctuation or symbol
  DS_SP = 7,   // U+0020
  DS_WS = 8,   // other \s but CR and LF
  DS_NL = 9,   // CR, LF
  DS_KL = 10,  // in the CJK/kana ranges: letter
  DS_KM = 11,  //   mark
  DS_KP = 12,  //   punctuation or symbol
  DS_KO = 13,  //   other
  DS_NONE = 15
};

// Class sets (bit c set when class c is in the set).
constexpr uint32_t DSM_LM = (1u << DS_AL) | (1u << DS_L) | (1u << DS_M) | (1u << DS_KL) | (1u << DS_KM);
constexpr uint32_t DSM_PS = (1u << DS_AP) | (1u << DS_PS) | (1u << DS_KP);
constexpr uint32_t DSM_SPACE = (1u << DS_SP) | (1u << DS_WS) | (1u << DS_NL);
// [^\r\n\p{L}\p{P}\p{S}]: D2's optional first character
constexpr uint32_t DSM_PFX =
    (1u << DS_O) | (1u << DS_M) | (1u << DS_N) | (1u << DS_SP) | (1u << DS_WS) | (1u << DS_KM) | (1u << DS_KO);

// Group of a class: 0 the rest, 1 numbers, 2 the CJK/kana set, 3 none.
__host__ __device__ inline uint32_t ds_group(uint32_t c) {
  return c == DS_N ? 1u : (c >= DS_KL && c <= DS_KO) ? 2u : c == DS_NONE ? 3u : 0u;
}

// Class of an ASCII code point (equal to the table's; computed, so that it
// does not depend on the table being staged yet).
__host__ __device__ inline uint32_t ds_ascii_class(uint32_t cp) {
  if (((cp | 32u) - 'a') < 26u) return DS_AL;
  if ((cp - '0') < 10u) return DS_N;
  if (cp == 10u || cp == 13u) return DS_NL;
  if (cp == 32u) return DS_SP;
  if (cp == 9u || cp == 11u || cp == 12u) return DS_WS;
  if ((cp - 33u) < 94u) return DS_AP;  // the printable characters left are punctuation and symbols
  return DS_O;
}

template <class P>
__host__ __device__ inline uint32_t ds_table_class(P l1, P l2, uint32_t cp) {
  const uint32_t blk = l1[cp >> 8];
  return (l2[blk * 128u + ((cp & 255u) >> 1)] >> ((cp & 1u) * 4u)) & 15u;
}

// Whether a position whose left character has class x and whose right
// character has class y is a synchronizing boundary of the DeepSeek-style
// pattern: every text with these two characters there has a piece boundary
// between them, the pieces to the right depend on the left only through x,
// and the pieces to the left depend on the right only through y.  A group
// change always is one.  Inside the rest, from the third splitter:
//   - before a letter or mark: after CR/LF, a number or a non-ASCII
//     punctuation mark or symbol (which can neither be D2's first character
//     nor take letters in D1); a non-ASCII letter or a mark also after ASCII
//     punctuation (D1 takes ASCII letters only);
//   - before punctuation or a symbol: after a letter, a mark, CR/LF, other
//     whitespace than U+0020 or a character of none of the classes;
//   - before whitespace: after a letter, a mark, punctuation, a symbol or a
//     character of none of the classes; before CR/LF not after punctuation or
//     a symbol (D3 takes CR/LF after them) nor after whitespace;
//   - before a character of none of the classes: after anything but another
//     such character (which may be D2's first character before letters).
// Inside the CJK/kana set: before a letter or mark, after punctuation or a
// symbol; before punctuation or a symbol, after anything else of the set
// (D3 does not take letters, marks or unassigned code points); before an
// unassigned code point, after anything but another one (which may be D2's
// first character before letters).
__host__ __device__ inline bool ds_sync(uint32_t x, uint32_t y) {
  if (x == DS_NONE || y == DS_NONE) return false;
  if (ds_group(x) != ds_group(y)) return true;
  const uint32_t bx = 1u << x;
  switch (y) {
    case DS_AL: return (bx & ((1u << DS_NL) | (1u << DS_PS))) != 0u;
    case DS_L:
    case DS_M: return (bx & ((1u << DS_NL) | (1u << DS_PS) | (1u << DS_AP))) != 0u;
    case DS_AP:
    case DS_PS:
      return (bx & ((1u << DS_AL) | (1u << DS_L) | (1u << DS_M) | (1u << DS_NL) | (1u << DS_O) | (1u << DS_WS))) != 0u;
    case DS_SP:
    case DS_WS: return (bx & ((1u << DS_AL) | (1u << DS_L) | (1u << DS_M) | (1u << DS_AP) | (1u << DS_PS) | (1u << DS_O))) != 0u;
    case DS_NL: return (bx & ((1u << DS_AL) | (1u << DS_L) | (1u << DS_M) | (1u << DS_O))) != 0u;
    case DS_O: return x != DS_O;
    case DS_KL:
    case DS_KM: return x == DS_KP;
    case DS_KP: return x != DS_KP;
    case DS_KO: return x != DS_KO;
    default: return false;
  }
}

// DeepSeek-style class of the character at window index q of a tile's view
// of the request (tt_o200k.h), outside the window from the text and the table.
__device__ inline uint32_t ds_view_cls(const O2View& v, int64_t q) {
  if (v.in_win(q)) return v.code[PT_PAD + q] & 15u;
  const uint32_t b0 = v.byte(q);
  if (b0 < 0x80u) return ds_table_class(v.l1, v.l2, b0);
  const uint32_t L = o2_lead_len(b0);
  if (L == 1u) return DS_NONE;
  uint32_t cp = b0 & (0x7Fu >> L);
  for (uint32_t k = 1; k < L; ++k) {
    if (v.w0 + q + k >= v.n) return DS_NONE;
    cp = (cp << 6) | (v.byte(q + k) & 0x3Fu);
  }
  return cp < 0x110000u ? ds_table_class(v.l1, v.l2, cp) : DS_NONE;
}

// Class of a character outside the window (rare: walks that run past it).
__device__ __noinline__ uint32_t ds_cls_far(const O2View v, int64_t q) { return ds_view_cls(v, q); }

// End (window index) of the piece that starts at s.  Always > s.  A piece
// of numbers is one to three of them (walks start at a number stretch's
// head, so the chunks line up with it).  Otherwise the third splitter runs
// inside the group stretch of s: its alternatives in order, and when none
// matches at s, the unmatched stretch up to the next position where one does.
__device__ __forceinline__ int64_t ds_piece_end(const O2View& v, int64_t s) {
  auto cls = [&](int64_t q) -> uint32_t { return v.in_win(q) ? (uint32_t)(v.code[PT_PAD + q] & 15u) : ds_cls_far(v, q); };
  const uint32_t c0 = cls(s);
  const uint32_t g0 = ds_group(c0);
  // q is beyond the group stretch of s (the third splitter's end of text)
  auto stop = [&](int64_t q) { return q > s && (v.past(q) || ds_group(cls(q)) != g0); };
  auto in = [&](int64_t q, uint32_t mask) { return !stop(q) && ((mask >> cls(q)) & 1u) != 0u; };
  auto scan = [&](int64_t q, uint32_t mask) -> int64_t {
    while (in(q, mask)) q += v.clen(q);
    return q;
  };
  const int64_t s1 = s + v.clen(s);
  if (c0 == DS_N) {  // S1
    int64_t q = s1;
    for (int k = 1; k < 3 && in(q, 1u << DS_N); ++k) q += v.clen(q);
    return q;
  }
  // D1: ASCII punctuation or symbol, then ASCII letters
  if (c0 == DS_AP && in(s1, 1u << DS_AL)) return scan(s1, 1u << DS_AL);
  // D2: the optional first character, then letters and marks
  if ((DSM_PFX >> c0) & 1u) {
    const int64_t e = scan(s1, DSM_LM);
    if (e > s1) return e;
  }
  if ((DSM_LM >> c0) & 1u) return scan(s1, DSM_LM);
  // D3: optional U+0020, punctuation and symbols, then CR/LF
  const int64_t st = (c0 == DS_SP && in(s1, DSM_PS)) ? s1 : s;
  if (in(st, DSM_PS)) return scan(scan(st, DSM_PS), 1u << DS_NL);
  // D4-D6: whitespace
  if ((DSM_SPACE >> c0) & 1u) {
    int64_t q = s, last_nl = -1, last_start = s;
    while (in(q, DSM_SPACE)) {
      if (cls(q) == DS_NL) last_nl = q;
      last_start = q;
      q += v.clen(q);
    }
    if (last_nl >= 0) return last_nl + 1;  // \s*[\r\n]+ (CR and LF are one byte)
    if (stop(q)) return q;                  // \s+(?!\S) at the end of the stretch
    return last_start > s ? last_start : q; // gives back the last character, else \s+
  }
  // no alternative matches at s: the unmatched stretch ends where one does,
  // which is any character but one of none of the classes that no letter or
  // mark follows
  int64_t q = s1;
  while (!stop(q)) {
    const uint32_t c = cls(q);
    if (c != DS_O && c != DS_KO) break;
    const int64_t q1 = q + v.clen(q);
    if (in(q1, DSM_LM)) break;
    q = q1;
  }
  return q;
}

}  // namespace tt
