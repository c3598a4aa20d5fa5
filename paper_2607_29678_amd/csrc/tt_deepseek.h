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
__host__ __device__ constexpr uint32_t ds_group(uint32_t c) {
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

// The DeepSeek-style bitmaps (run sets, tt_o200k.h): numbers; ASCII
// letters; letters and marks of the rest; letters and marks of the CJK/kana
// set; punctuation and symbols of the rest; those of the CJK/kana set;
// whitespace; and CR/LF (single bytes: their bitmap serves runs and "last").
// A set never mixes the groups, so a run stops at a group change.
enum : int { DSB_N = 0, DSB_AL = 1, DSB_LM0 = 2, DSB_LM2 = 3, DSB_PS0 = 4, DSB_PS2 = 5, DSB_SP = 6, DSB_NL = 7 };
constexpr uint32_t DSB_RUNS = (1u << DSB_N) | (1u << DSB_AL) | (1u << DSB_LM0) | (1u << DSB_LM2) | (1u << DSB_PS0) |
                              (1u << DSB_PS2) | (1u << DSB_SP);
__host__ __device__ constexpr uint32_t ds_bits_of(uint32_t c) {
  switch (c) {
    case DS_N: return 1u << DSB_N;
    case DS_AL: return (1u << DSB_AL) | (1u << DSB_LM0);
    case DS_L:
    case DS_M: return 1u << DSB_LM0;
    case DS_KL:
    case DS_KM: return 1u << DSB_LM2;
    case DS_AP:
    case DS_PS: return 1u << DSB_PS0;
    case DS_KP: return 1u << DSB_PS2;
    case DS_SP:
    case DS_WS: return 1u << DSB_SP;
    case DS_NL: return (1u << DSB_SP) | (1u << DSB_NL);
    default: return 0u;
  }
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
__host__ __device__ constexpr bool ds_sync(uint32_t x, uint32_t y) {
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

// Branch-free forms of ds_sync and ds_bits_of for the tile kernel, as bit
// tables built from the functions themselves: ds_sync in four 64-bit tables
// (table y / 4, bit 16 (y % 4) + x), and per bitmap the classes in it.
constexpr uint64_t ds_sync_table(uint32_t yq) {
  uint64_t t = 0;
  for (uint32_t y = 4 * yq; y < 4 * yq + 4; ++y)
    for (uint32_t x = 0; x < 16; ++x)
      if (ds_sync(x, y)) t |= 1ull << (16 * (y - 4 * yq) + x);
  return t;
}
__device__ __forceinline__ bool ds_sync_bits(uint32_t x, uint32_t y) {
  constexpr uint64_t T0 = ds_sync_table(0), T1 = ds_sync_table(1), T2 = ds_sync_table(2), T3 = ds_sync_table(3);
  const uint32_t yq = y >> 2;
  const uint64_t t = yq == 0u ? T0 : yq == 1u ? T1 : yq == 2u ? T2 : T3;
  return ((t >> (16u * (y & 3u) + (x & 15u))) & 1u) != 0u;
}
constexpr uint32_t ds_bitmap_classes(int k) {
  uint32_t m = ((DSB_RUNS >> k) & 1u) << DS_NONE;
  for (uint32_t c = 0; c < 15; ++c)
    if ((ds_bits_of(c) >> k) & 1u) m |= 1u << c;
  return m;
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

// The classes of a group (bit c set when class c is in it): the rest, and
// the CJK/kana set.
constexpr uint32_t DSM_G0 = (1u << DS_O) | (1u << DS_AL) | (1u << DS_L) | (1u << DS_M) | (1u << DS_AP) |
                            (1u << DS_PS) | (1u << DS_SP) | (1u << DS_WS) | (1u << DS_NL);
constexpr uint32_t DSM_G2 = (1u << DS_KL) | (1u << DS_KM) | (1u << DS_KP) | (1u << DS_KO);

// The class set of run bitmap k (its classes of one group), and the classes
// whose last character the scans of that set track.
__host__ __device__ inline uint32_t ds_run_mask(int k) {
  return k == DSB_N ? 1u << DS_N : k == DSB_AL ? 1u << DS_AL : k == DSB_LM0 ? DSM_LM & DSM_G0
         : k == DSB_LM2 ? DSM_LM & DSM_G2 : k == DSB_PS0 ? DSM_PS & DSM_G0 : k == DSB_PS2 ? DSM_PS & DSM_G2
         : k == DSB_SP ? DSM_SPACE : k == DSB_NL ? 1u << DS_NL : 0u;
}
__host__ __device__ inline uint32_t ds_run_track(int k) { return k == DSB_SP ? 1u << DS_NL : 0u; }

// The part of a run scan past the window (rare), as scan_far in tt_o200k.h,
// with `mask` holding classes of one group only.
__device__ __noinline__ ScanEnd ds_scan_far(const O2View v, int64_t q, uint32_t mask, uint32_t track, int64_t last) {
  return scan_far(v, q, mask, track, last, [&](uint32_t cp) { return ds_table_class(v.l1, v.l2, cp); });
}

// far_serve for the DeepSeek-style pattern, out of line.
__device__ __noinline__ void ds_far_serve(const O2View v, uint32_t sets) {
  far_serve(v, sets, ds_run_mask, ds_run_track, [&](uint32_t cp) { return ds_table_class(v.l1, v.l2, cp); });
}

// End (window index) of the piece that starts at s.  Always > s.  A piece
// of numbers is one to three of them (walks start at a number stretch's
// head, so the chunks line up with it).  Otherwise the third splitter runs
// inside the group stretch of s: its alternatives in order, and when none
// matches at s, the unmatched stretch up to the next position where one does.
// The alternatives that match end with a run scan (one for letters, one for
// whitespace, two for punctuation then CR/LF).  The view is one of those of
// tt_o200k.h.
template <class V, class P>
__device__ __forceinline__ P ds_end(V& v, const P s) {
  const uint32_t c0 = v.cls(s);
  const uint32_t g0 = ds_group(c0);
  const uint32_t gm = g0 == 0u ? DSM_G0 : g0 == 2u ? DSM_G2 : 0u;
  // q is beyond the group stretch of s (the third splitter's end of text)
  auto stop = [&](P q) { return q > s && (v.past(q) || ds_group(v.cls(q)) != g0); };
  auto in = [&](P q, uint32_t mask) { return !stop(q) && ((mask >> v.cls(q)) & 1u) != 0u; };
  const P s1 = s + (P)v.clen(s);
  if (c0 == DS_N) {  // S1
    P q = s1;
    for (int k = 1; k < 3 && in(q, 1u << DS_N); ++k) q += (P)v.clen(q);
    return q;
  }
  // the closing run (run bitmaps hold the classes of one group, and the
  // classes passed for the part past the window are those of the group of s)
  int alt;
  P q0 = s1, last = -1;
  uint32_t mask, track = 0u;
  int rb, tb = -1;
  if (c0 == DS_AP && in(s1, 1u << DS_AL)) {
    // D1: ASCII punctuation or symbol, then ASCII letters
    alt = 1;
    mask = 1u << DS_AL;
    rb = DSB_AL;
  } else if (((DSM_LM >> c0) & 1u) || (((DSM_PFX >> c0) & 1u) && in(s1, DSM_LM))) {
    // D2: the optional first character, then letters and marks
    alt = 1;
    mask = DSM_LM;
    rb = g0 == 2u ? DSB_LM2 : DSB_LM0;
  } else {
    // D3: optional U+0020, punctuation and symbols, then CR/LF
    const P st = (c0 == DS_SP && in(s1, DSM_PS)) ? s1 : s;
    if (in(st, DSM_PS)) {
      alt = 3;
      q0 = st + (P)v.clen(st);
      mask = DSM_PS;
      rb = g0 == 2u ? DSB_PS2 : DSB_PS0;
    } else if ((DSM_SPACE >> c0) & 1u) {
      // D4-D6: whitespace, with its last CR/LF
      alt = 4;
      mask = DSM_SPACE;
      track = 1u << DS_NL;
      rb = DSB_SP;
      tb = DSB_NL;
      if (c0 == DS_NL) last = s;
    } else {
      // no alternative matches at s: the unmatched stretch ends where one
      // does, which is any character but one of none of the classes that no
      // letter or mark follows
      P q = s1;
      while (!stop(q)) {
        const uint32_t c = v.cls(q);
        if (c != DS_O && c != DS_KO) break;
        const P q1 = q + (P)v.clen(q);
        if (in(q1, DSM_LM)) break;
        q = q1;
      }
      return q;
    }
  }
  P e;
#pragma unroll 1
  for (;;) {
    e = v.scan(q0, mask & gm, track, last, rb, tb);
    if (alt != 3 || g0 != 0u) break;
    alt = 1;  // D3 in the rest: then CR/LF (in the CJK/kana set there is none)
    q0 = e;
    mask = 1u << DS_NL;
    rb = DSB_NL;
  }
  if (alt != 4) return e;
  if (last >= 0) return last + 1;  // \s*[\r\n]+ (CR and LF are one byte)
  if (stop(e)) return e;           // \s+(?!\S) at the end of the stretch
  // \s+(?!\S) gives back the last character, if there are two or more
  for (P r = e - 1; r > s && r >= e - 4; --r)
    if ((v.byte(r) & 0xC0u) != 0x80u) return r;
  return e;  // else \s+
}

// The piece's end with the full view (rare: pieces at the window's end), or
// -1 - k when the run through the window's end of bitmap k is needed first.
__device__ __noinline__ int64_t ds_end_full(const O2View v, int64_t s) {
  FullView<ds_cls_far, ds_scan_far> f{v};
  const int64_t e = ds_end(f, s);
  return f.need >= 0 ? -1 - (int64_t)f.need : e;
}

// End (window index) of the piece that starts at s (0 <= s < PT_WIN), or
// -1 - k as ds_end_full.
__device__ __forceinline__ int64_t ds_piece_end(const O2View& v, int64_t s) {
  WinView f{v.buf, v.code, v.bits, (int32_t)(v.n - v.w0 < PT_WIN ? v.n - v.w0 : PT_WIN)};
  const int32_t e = ds_end(f, (int32_t)s);
  if (!f.out && e + WIN_MARGIN <= PT_WIN) return e;
  return ds_end_full(v, s);
}

}  // namespace tt
