// Incremental repair: a session keeps the text of a growing request and the
// records of its full tokenization, and an append re-tokenizes only a window
// at the end (Sec. 3.2, "Incremental repair"; Sec. 3.4 keeps the records in
// arrays that are edited in place, so an append costs O(append + window)).
//
// Why a splice is exact (Appendix, "The Splice Theorem"): tokenization is
// pre-tokenization into pieces followed by per-piece BPE (Lemma l:homo).  If
// a byte position p is a piece boundary of the whole text A ++ B, of A alone
// and of the window, the pieces left of p agree between A and A ++ B, and the
// pieces right of p agree between the window and A ++ B, then the cached
// tokens left of p followed by the fresh tokens right of p are the tokens of
// A ++ B (Definition d:cert, Theorem t:main).  A synchronizing class
// transition gives all of this at once (sync_at below).  The deployed check
// looks for such a transition inside the longest run of records on which the
// cached and the fresh tokenization agree, and splices at the end of the run
// (Corollary c:shift: records coincide between the boundary and the end of
// the run).
//
// Everything here is host code; the windows are tokenized by the library's
// span export on the caller's stream, through pinned buffers with one
// synchronisation per window.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <vector>

#define TT_CLS_STORAGE static
#include "class_table.inc"
#include "class_table_o200k.inc"
#include "class_table_deepseek.inc"
#include "tt_internal.h"
#include "tt_deepseek.h"
#include "tt_o200k.h"

namespace {

// ---- character classes on the host ----------------------------------------
enum HostClass : int { H_O = 0, H_L = 1, H_N = 2, H_WS = 3, H_NL = 4 };

int host_class(uint32_t cp) {
  if (cp == 10u || cp == 13u) return H_NL;
  const uint32_t blk = TT_CLS_L1[cp >> 8];
  const uint32_t c2 = (TT_CLS_L2[blk * 64u + ((cp & 255u) >> 2)] >> ((cp & 3u) * 2u)) & 3u;
  return c2 == 1u ? H_L : c2 == 2u ? H_N : c2 == 3u ? H_WS : H_O;
}

// Strict UTF-8 decode of the character starting at s[i] (bytes [i, n)).
// Returns its length, or 0 if the bytes there are not a valid character.
int decode_at(const uint8_t* s, int64_t n, int64_t i, uint32_t& cp) {
  if (i < 0 || i >= n) return 0;
  const uint32_t b0 = s[i];
  int len = b0 < 0x80u ? 1 : b0 < 0xC2u ? 0 : b0 < 0xE0u ? 2 : b0 < 0xF0u ? 3 : b0 < 0xF5u ? 4 : 0;
  if (len == 0 || i + len > n) return 0;
  if (len == 1) {
    cp = b0;
    return 1;
  }
  const uint32_t b1 = s[i + 1];
  const uint32_t lo = b0 == 0xE0u ? 0xA0u : b0 == 0xF0u ? 0x90u : 0x80u;
  const uint32_t hi = b0 == 0xEDu ? 0x9Fu : b0 == 0xF4u ? 0x8Fu : 0xBFu;
  if (b1 < lo || b1 > hi) return 0;
  uint32_t c = b0 & (0x7Fu >> len);
  c = (c << 6) | (b1 & 0x3Fu);
  for (int k = 2; k < len; ++k) {
    const uint32_t b = s[i + k];
    if ((b & 0xC0u) != 0x80u) return 0;
    c = (c << 6) | (b & 0x3Fu);
  }
  cp = c;
  return len;
}

// Whether byte position p (0 < p < n) is a synchronizing boundary: the
// characters on either side of it form a transition of the pattern's set.
// The sets follow from the run-local rules of the two patterns (Sec. 4.1):
//
// GPT-2.  A run head starts a piece unless the character before it is U+0020
// (which then begins the piece) or it is the suffix letter of a contraction
// (an apostrophe before it).  The rules of a position look back at most to
// the apostrophe of a contraction and the character before that, and ahead
// only to see whether a whitespace run ends at a non-space character.  So at
// a change of class (whitespace counted as one class) whose left character is
// neither U+0020 nor an apostrophe, every text has a piece boundary, the
// decisions to the right see only the left character's class, and those to
// the left see only the right character's class.
//
// cl100k.  A number run head always starts a piece and numbers are grouped
// from the head.  A letter run head starts a piece unless a whitespace
// character other than CR/LF, a lone symbol or a contraction apostrophe
// precedes it, so only a number or CR/LF on its left is safe.  A symbol run
// head starts a piece unless U+0020 precedes it.  A whitespace run head
// starts a piece unless a symbol piece absorbs it (CR/LF after a symbol), and
// the pieces of a whitespace run depend on the run itself and on whether a
// symbol precedes it, so a run head is safe after a letter or number (and
// after a symbol when the head is not CR/LF), but a change between CR/LF and
// other whitespace is not.
//
// o200k: see o2_sync.  DeepSeek: see ds_sync.
bool sync_at(int pattern, const uint8_t* s, int64_t n, int64_t p) {
  if (p <= 0 || p >= n) return false;
  uint32_t cr = 0, cl = 0;
  if (decode_at(s, n, p, cr) == 0) return false;
  int64_t q = p - 1;  // lead byte of the character before p
  while (q > 0 && p - q < 4 && (s[q] & 0xC0u) == 0x80u) --q;
  if (decode_at(s, n, q, cl) != (int)(p - q)) return false;
  if (pattern == TT_PATTERN_DEEPSEEK)
    return tt::ds_sync(tt::ds_table_class(TT_DS_L1, TT_DS_L2, cl), tt::ds_table_class(TT_DS_L1, TT_DS_L2, cr));
  if (pattern == TT_PATTERN_O200K)
    return tt::o2_sync(tt::o2_table_class(TT_O2_L1, TT_O2_L2, cl), tt::o2_table_class(TT_O2_L1, TT_O2_L2, cr), cl, cr);
  const int x = host_class(cl), y = host_class(cr);
  const bool x_sp = cl == 0x20u, x_apo = cl == 0x27u;
  if (pattern == TT_PATTERN_GPT2) {
    auto merged = [](int c) { return c == H_NL ? H_WS : c; };
    return merged(x) != merged(y) && !x_sp && !x_apo;
  }
  switch (y) {
    case H_N: return x != H_N;
    case H_L: return x == H_N || x == H_NL;
    case H_O: return x == H_L || x == H_N || x == H_NL || (x == H_WS && !x_sp);
    case H_WS: return x == H_L || x == H_N || x == H_O;
    default: return x == H_L || x == H_N;  // H_NL
  }
}

// The decision for one window; see tt_splice_plan in the header.
struct Plan {
  bool accept = false;
  int64_t keep_c = 0, from_f = 0;
};

Plan plan_splice(int pattern, const uint8_t* text, int64_t len, int64_t a_len, int64_t x, const int32_t* c_ids,
                 const int32_t* c_spans, int64_t n_c, const int32_t* f_ids, const int32_t* f_spans, int64_t n_f,
                 int64_t max_token_chars) {
  Plan plan;
  // cached records that start inside the window (byte begins increase)
  int64_t i = 0;
  {
    int64_t lo = 0, hi = n_c;
    while (lo < hi) {
      const int64_t mid = (lo + hi) / 2;
      if (c_spans[4 * mid] < x) lo = mid + 1;
      else hi = mid;
    }
    i = lo;
  }
  // the longest run of aligned records that agree in byte span and ID (the
  // later one among equally long runs)
  int64_t j = 0, cur = 0, cur_i0 = 0, cur_j0 = 0;
  int64_t best = 0, best_i0 = 0, best_j0 = 0;
  while (i < n_c && j < n_f) {
    const int32_t cb = c_spans[4 * i], fb = f_spans[4 * j];
    if (cb == fb) {
      if (c_spans[4 * i + 1] == f_spans[4 * j + 1] && c_ids[i] == f_ids[j]) {
        if (cur == 0) {
          cur_i0 = i;
          cur_j0 = j;
        }
        ++cur;
        if (cur >= best) {
          best = cur;
          best_i0 = cur_i0;
          best_j0 = cur_j0;
        }
      } else {
        cur = 0;
      }
      ++i;
      ++j;
    } else if (cb < fb) {
      cur = 0;
      ++i;
    } else {
      cur = 0;
      ++j;
    }
  }
  // the stable boundary check
  if (best < 2) return plan;
  const int64_t i1 = best_i0 + best - 1;
  if ((int64_t)c_spans[4 * i1 + 3] - (int64_t)c_spans[4 * best_i0 + 2] <= max_token_chars) return plan;
  bool cert = false;
  for (int64_t k = best_i0; k <= i1 && !cert; ++k) {
    const int64_t p = c_spans[4 * k];
    cert = p > x && p < a_len && sync_at(pattern, text, len, p);
  }
  if (!cert) return plan;
  plan.accept = true;
  plan.keep_c = i1 + 1;
  plan.from_f = best_j0 + best;
  return plan;
}

}  // namespace

struct tt_session {
  tt_tokenizer* h = nullptr;
  int pattern = 0;
  int64_t w0 = 512;               // first window, characters
  int64_t max_tok_chars = 1;      // the check's length bound
  std::vector<uint8_t> text;
  int64_t n_chars = 0;
  std::vector<int32_t> ids;       // records of the full tokenization of `text`
  std::vector<int32_t> spans;     // 4 per token, text coordinates
  std::vector<int32_t> f_ids, f_spans;  // records of a whole-text tokenization
  // windows go through pinned buffers (one synchronisation per window)
  int64_t pin_cap = 0;
  uint8_t* p_in = nullptr;
  int32_t* p_ids = nullptr;
  int32_t* p_spans = nullptr;
  int64_t* p_len = nullptr;

  ~tt_session() {
    if (p_in) (void)hipHostFree(p_in);
    if (p_ids) (void)hipHostFree(p_ids);
    if (p_spans) (void)hipHostFree(p_spans);
    if (p_len) (void)hipHostFree(p_len);
  }
};

namespace {

int64_t count_chars(const uint8_t* s, int64_t n) {
  int64_t c = 0;
  for (int64_t i = 0; i < n; ++i) c += (s[i] & 0xC0u) != 0x80u;
  return c;
}

constexpr int64_t PIN_MAX = 1 << 20;  // largest window staged in pinned memory (bytes)

int grow_pinned(tt_session* s, int64_t n) {
  if (n <= s->pin_cap) return TT_OK;
  int64_t cap = 65536;
  while (cap < n) cap <<= 1;
  if (s->p_in) (void)hipHostFree(s->p_in);
  if (s->p_ids) (void)hipHostFree(s->p_ids);
  if (s->p_spans) (void)hipHostFree(s->p_spans);
  s->p_in = nullptr;
  s->p_ids = nullptr;
  s->p_spans = nullptr;
  s->pin_cap = 0;
  if (!s->p_len && hipHostMalloc(reinterpret_cast<void**>(&s->p_len), 8, hipHostMallocDefault) != hipSuccess)
    return TT_ERR_OOM;
  if (hipHostMalloc(reinterpret_cast<void**>(&s->p_in), (size_t)cap, hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc(reinterpret_cast<void**>(&s->p_ids), 4 * (size_t)cap, hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc(reinterpret_cast<void**>(&s->p_spans), 16 * (size_t)cap, hipHostMallocDefault) != hipSuccess)
    return TT_ERR_OOM;
  s->pin_cap = cap;
  return TT_OK;
}

// Records of text[from, end) with spans shifted to text coordinates, in
// *ids / *spans (the session's pinned buffers for a window, its vectors for a
// longer range); returns the token count or an error.
int64_t encode_range(tt_session* s, int64_t from, int64_t chars_before, void* stream, int32_t** ids,
                     int32_t** spans) {
  const int64_t n = (int64_t)s->text.size() - from;
  int64_t T = 0;
  if (n <= PIN_MAX) {
    int rc = grow_pinned(s, n);
    if (rc != TT_OK) return rc;
    std::memcpy(s->p_in, s->text.data() + from, (size_t)n);
    rc = tt::encode_spans_pinned(s->h, s->p_in, n, s->p_ids, s->p_spans, s->p_len, stream);
    if (rc != TT_OK) return rc;
    T = *s->p_len;
    *ids = s->p_ids;
    *spans = s->p_spans;
  } else {
    s->f_ids.resize((size_t)n);
    s->f_spans.resize(4 * (size_t)n);
    const int rc = tt_encode_spans(s->h, s->text.data() + from, n, s->f_ids.data(), s->f_spans.data(), &T, stream);
    if (rc != TT_OK) return rc;
    *ids = s->f_ids.data();
    *spans = s->f_spans.data();
  }
  if (from != 0) {
    int32_t* sp = *spans;
    for (int64_t k = 0; k < T; ++k) {
      sp[4 * k] += (int32_t)from;
      sp[4 * k + 1] += (int32_t)from;
      sp[4 * k + 2] += (int32_t)chars_before;
      sp[4 * k + 3] += (int32_t)chars_before;
    }
  }
  return T;
}

}  // namespace

extern "C" {

int tt_sync_boundaries(int32_t pattern_id, const uint8_t* utf8, int64_t len, uint8_t* out_mask) {
  if (len < 0) return TT_ERR_BAD_ARG;
  if (len > 0 && (!utf8 || !out_mask)) return TT_ERR_NULL_ARG;
  if (pattern_id != TT_PATTERN_GPT2 && pattern_id != TT_PATTERN_CL100K && pattern_id != TT_PATTERN_O200K &&
      pattern_id != TT_PATTERN_DEEPSEEK) return TT_ERR_BAD_PATTERN;
  for (int64_t p = 0; p < len; ++p) out_mask[p] = sync_at(pattern_id, utf8, len, p) ? 1 : 0;
  return TT_OK;
}

int tt_splice_plan(int32_t pattern_id, const uint8_t* text, int64_t len, int64_t a_len, int64_t x,
                   const int32_t* c_ids, const int32_t* c_spans, int64_t n_c, const int32_t* f_ids,
                   const int32_t* f_spans, int64_t n_f, int64_t max_token_chars, int64_t* keep_c,
                   int64_t* from_f) {
  if (!text || !keep_c || !from_f || (n_c > 0 && (!c_ids || !c_spans)) || (n_f > 0 && (!f_ids || !f_spans)))
    return TT_ERR_NULL_ARG;
  if (pattern_id != TT_PATTERN_GPT2 && pattern_id != TT_PATTERN_CL100K && pattern_id != TT_PATTERN_O200K &&
      pattern_id != TT_PATTERN_DEEPSEEK) return TT_ERR_BAD_PATTERN;
  if (len <= 0 || a_len <= 0 || a_len > len || x <= 0 || x >= a_len || n_c < 0 || n_f < 0 || len > TT_MAX_BYTES)
    return TT_ERR_BAD_ARG;
  const Plan p = plan_splice(pattern_id, text, len, a_len, x, c_ids, c_spans, n_c, f_ids, f_spans, n_f,
                             max_token_chars);
  if (!p.accept) return 0;
  *keep_c = p.keep_c;
  *from_f = p.from_f;
  return 1;
}

int tt_session_create(tt_tokenizer* h, int32_t window_chars, tt_session** out) {
  if (!h || !out) return TT_ERR_NULL_ARG;
  *out = nullptr;
  if (window_chars < 0 || tt::handle_has_added(h)) return TT_ERR_BAD_ARG;
  tt_session* s = new tt_session();
  s->h = h;
  s->pattern = tt::handle_pattern(h);
  s->w0 = window_chars > 0 ? window_chars : 512;
  // a token spells at most as many characters as it has bytes
  s->max_tok_chars = (int64_t)tt::handle_max_token_bytes(h);
  *out = s;
  return TT_OK;
}

void tt_session_destroy(tt_session* s) { delete s; }

int tt_session_append(tt_session* s, const uint8_t* utf8, int64_t len, tt_append_info* info, void* stream) {
  if (!s || (len > 0 && !utf8)) return TT_ERR_NULL_ARG;
  if (len < 0) return TT_ERR_BAD_ARG;
  const int64_t a_len = (int64_t)s->text.size();
  const int64_t T_old = (int64_t)s->ids.size();
  tt_append_info r{T_old, T_old, 0, 0, 0};
  if (len == 0) {
    if (info) *info = r;
    return TT_OK;
  }
  if (a_len + len > TT_MAX_BYTES) return TT_ERR_TOO_LARGE;
  // the new text, kept only if the append succeeds
  s->text.insert(s->text.end(), utf8, utf8 + len);
  const int64_t n = (int64_t)s->text.size();
  const uint8_t* t = s->text.data();
  auto fail = [&](int rc) {
    s->text.resize((size_t)a_len);
    return rc;
  };
  int32_t *f_ids = nullptr, *f_spans = nullptr;
  bool done = false;
  if (a_len > 0) {
    for (int attempt = 0; attempt <= 5 && !done; ++attempt) {
      const int64_t w = s->w0 << attempt;
      // the window starts w characters before the end of A
      int64_t x = a_len, c = 0;
      while (x > 0 && c < w) {
        --x;
        c += (t[x] & 0xC0u) != 0x80u;
      }
      if (x == 0) break;  // the window reaches the text start: tokenize the whole text
      const int64_t T = encode_range(s, x, s->n_chars - w, stream, &f_ids, &f_spans);
      if (T < 0) return fail((int)T);
      ++r.windows;
      const Plan p = plan_splice(s->pattern, t, n, a_len, x, s->ids.data(), s->spans.data(), T_old, f_ids,
                                 f_spans, T, s->max_tok_chars);
      if (!p.accept) continue;
      // in place: drop the cached tail, append the fresh records after the run
      s->ids.resize((size_t)p.keep_c);
      s->spans.resize(4 * (size_t)p.keep_c);
      s->ids.insert(s->ids.end(), f_ids + p.from_f, f_ids + T);
      s->spans.insert(s->spans.end(), f_spans + 4 * p.from_f, f_spans + 4 * T);
      r.kept = p.keep_c;
      r.window_chars = w;
      done = true;
    }
  }
  if (!done) {  // the whole text
    const int64_t T = encode_range(s, 0, 0, stream, &f_ids, &f_spans);
    if (T < 0) return fail((int)T);
    s->ids.assign(f_ids, f_ids + T);
    s->spans.assign(f_spans, f_spans + 4 * T);
    r.kept = 0;
    r.full = 1;
  }
  s->n_chars += count_chars(utf8, len);
  r.n_tokens = (int64_t)s->ids.size();
  if (info) *info = r;
  return TT_OK;
}

int tt_session_tokens(const tt_session* s, int64_t from, int64_t count, int32_t* out_ids, int32_t* out_spans) {
  if (!s) return TT_ERR_NULL_ARG;
  const int64_t T = (int64_t)s->ids.size();
  if (from < 0 || count < 0 || from > T || count > T - from) return TT_ERR_BAD_ARG;
  if (count == 0) return TT_OK;
  if (out_ids) std::memcpy(out_ids, s->ids.data() + from, 4 * (size_t)count);
  if (out_spans) std::memcpy(out_spans, s->spans.data() + 4 * from, 16 * (size_t)count);
  return TT_OK;
}

int tt_session_info(const tt_session* s, int64_t* n_bytes, int64_t* n_chars, int64_t* n_tokens) {
  if (!s) return TT_ERR_NULL_ARG;
  if (n_bytes) *n_bytes = (int64_t)s->text.size();
  if (n_chars) *n_chars = s->n_chars;
  if (n_tokens) *n_tokens = (int64_t)s->ids.size();
  return TT_OK;
}

}  // extern "C"
