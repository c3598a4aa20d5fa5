/*
 * toktier.h — C ABI of the exact GPU tokenizer for AMD Instinct MI355X (gfx950).
 *
 * The library computes, on one GPU, the full-request tokenization path of
 * "TokTier: Exact Stateful CPU+GPU Tokenization for Agentic LLM Serving":
 * exact GPT-family regex pre-tokenization recast as run-local rules
 * (Sec. 4.1, "Removing the sequential regex scan"), then exact byte-level BPE
 * (Sec. 4.2, "GPU BPE"), with output compaction.  The output contract is the
 * paper's (Sec. 1; Sec. 3 problem statement): the emitted token IDs are
 * identical to full reference tokenization of the whole request, i.e. to
 * leftmost-first pre-tokenization followed by per-piece greedy lowest-rank
 * BPE (Appendix, Definition d:frontend and Lemma l:homo).  No floating point
 * is involved.
 *
 * Conventions
 *  - All sizes are int64_t; token IDs are int32_t.
 *  - "host" pointers are ordinary CPU memory (pinned memory is faster but not
 *    required); "device" pointers are HIP device memory of the current device.
 *  - `stream` is a hipStream_t passed as void*; NULL means the null stream.
 *    All work of a call is enqueued on that stream.
 *  - Every function returns TT_OK (0) or a negative TT_ERR_* code.  On error
 *    nothing is written to caller buffers except where stated.
 *  - Byte-level BPE emits at most one ID per input byte, so an output buffer
 *    of `len` IDs (or the total byte count for a batch) is always enough.
 *  - A handle is immutable after tt_create (Sec. 4.5: registry entries are
 *    immutable after registration).  Calls on one handle from several host
 *    threads are allowed if each thread uses its own stream; the handle keeps
 *    one workspace per stream.
 *  - Memory: a stream's workspace takes about 35 bytes of device memory per
 *    byte of request capacity (epoch-tagged tile words, staging of tokens,
 *    rows of long units, the request bytes and IDs of host calls).  Host
 *    calls of tt_encode_spans add 16 bytes of device memory per byte, and
 *    host calls of tt_encode 5 bytes of pinned host memory per byte.  The
 *    capacity grows in powers of two from 64 KiB to the largest request seen
 *    on the stream (about 37 GB of device memory at TT_MAX_BYTES) and is freed
 *    by tt_destroy.
 */
#ifndef TOKTIER_H
#define TOKTIER_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------- */
enum {
  TT_OK = 0,
  TT_ERR_NULL_ARG = -1,     /* a required pointer is NULL                         */
  TT_ERR_BAD_PATTERN = -2,  /* pattern_id is not a TT_PATTERN_* value             */
  TT_ERR_BAD_MERGES = -3,   /* merge table out of range, duplicated or not proper */
  TT_ERR_BAD_VOCAB = -4,    /* vocabulary inconsistent with the merges            */
  TT_ERR_INVALID_UTF8 = -5, /* input is not strict UTF-8                          */
  TT_ERR_TOO_LARGE = -6,    /* request larger than TT_MAX_BYTES                   */
  TT_ERR_HIP = -7,          /* a HIP runtime call failed                          */
  TT_ERR_OOM = -8,          /* device or pinned host allocation failed            */
  TT_ERR_BAD_ARG = -9       /* a size or offset argument is inconsistent          */
};

/* Largest request (or batch) in bytes.  Offsets are kept in 32-bit words on
 * the device. */
#define TT_MAX_BYTES ((int64_t)1 << 30)

/* ---- pattern families ------------------------------------------------ */
/* Pre-tokenization pattern, each a leftmost-first alternation (Sec. 4.1):
 *  TT_PATTERN_GPT2:   's 't 're 've 'm 'll 'd | ?\p{L}+ | ?\p{N}+ |
 *                      ?[^\s\p{L}\p{N}]+ | \s+(?!\S) | \s+
 *  TT_PATTERN_CL100K: (?i:'s|'t|'re|'ve|'m|'ll|'d) | [^\r\n\p{L}\p{N}]?\p{L}+ |
 *                     \p{N}{1,3} | ?[^\s\p{L}\p{N}]+[\r\n]* | \s*[\r\n]+ |
 *                     \s+(?!\S) | \s+
 *  TT_PATTERN_O200K:  [^\r\n\p{L}\p{N}]?[\p{Lu}\p{Lt}\p{Lm}\p{Lo}\p{M}]*[\p{Ll}\p{Lm}\p{Lo}\p{M}]+CT? |
 *                     [^\r\n\p{L}\p{N}]?[\p{Lu}\p{Lt}\p{Lm}\p{Lo}\p{M}]+[\p{Ll}\p{Lm}\p{Lo}\p{M}]*CT? |
 *                     \p{N}{1,3} | ?[^\s\p{L}\p{N}]+[\r\n/]* | \s*[\r\n]+ | \s+(?!\S) | \s+
 *                     with CT = (?i:'s|'t|'re|'ve|'m|'ll|'d) (Sec. 4.1: the o200k lineage's
 *                     case boundaries; marks are letter material here)
 *  TT_PATTERN_DEEPSEEK: three splitters in sequence, each re-splitting every piece of the
 *                     one before, unmatched stretches kept as pieces (Sec. 4.1, the DeepSeek
 *                     family): \p{N}{1,3}; then [\u4E00-\u9FA5\u3040-\u309F\u30A0-\u30FF]+;
 *                     then [ASCII punctuation or symbol][A-Za-z]+ |
 *                     [^\r\n\p{L}\p{P}\p{S}]?[\p{L}\p{M}]+ | ?[\p{P}\p{S}]+[\r\n]* |
 *                     \s*[\r\n]+ | \s+(?!\S) | \s+
 * Character classes are those of the Oniguruma engine of HF tokenizers 0.22.2
 * (the paper pins class tables probed from the reference engine, Sec. 4.1). */
enum { TT_PATTERN_GPT2 = 0, TT_PATTERN_CL100K = 1, TT_PATTERN_O200K = 2, TT_PATTERN_DEEPSEEK = 3 };

typedef struct tt_tokenizer tt_tokenizer; /* opaque */

/* One BPE merge: the adjacent pair (left, right) becomes `result`.  In a merge
 * array the index is the rank: index 0 is applied first. */
typedef struct {
  int32_t left, right, result;
} tt_merge;

/* ---- create / destroy ------------------------------------------------ */
/* Build an immutable tokenizer handle on the current HIP device.
 *
 *  merges[n_merges]          rank-ordered merge list (host).
 *  vocab_bytes, vocab_offsets  token i is vocab_bytes[vocab_offsets[i] ..
 *                            vocab_offsets[i+1]) (host; offsets has
 *                            vocab_size+1 entries, non-decreasing, from 0).
 *  pattern_id                TT_PATTERN_GPT2, TT_PATTERN_CL100K, TT_PATTERN_O200K
 *                            or TT_PATTERN_DEEPSEEK.
 *  out                       receives the handle.
 *
 * The base ID of byte b is the lowest ID whose vocabulary entry is the single
 * byte b; all 256 must exist.  The merge list must be *proper*, which is what
 * makes one round of merging all leftmost non-overlapping occurrences of the
 * lowest-ranked pair equal to merging them one at a time (Sec. 4.2):
 *   - left, right, result lie in [0, vocab_size); no pair occurs twice;
 *   - each operand of merge r is a base ID or the result of a merge of rank < r;
 *   - results are pairwise distinct and none is a base ID;
 *   - vocab[result] == vocab[left] ++ vocab[right].
 * Violations return TT_ERR_BAD_MERGES (ranges, duplicates, properness) or
 * TT_ERR_BAD_VOCAB (byte strings, missing single bytes).  All inputs are
 * copied; the caller may free them on return.  Device tables live until
 * tt_destroy. */
int tt_create(const tt_merge* merges, int32_t n_merges, const uint8_t* vocab_bytes,
              const int64_t* vocab_offsets, int32_t vocab_size, int32_t pattern_id,
              tt_tokenizer** out);

/* Front-end options of tt_create_ex. */
typedef struct {
  /* 1: the model stage probes the vocabulary first and a piece that is a
   * vocabulary entry becomes that entry's single ID, without merging
   * (Sec. 4.2: families configured with ignore_merges).  Where several IDs
   * spell the same bytes the lowest is taken. */
  int32_t ignore_merges;
  /* Added tokens: literal strings that the model reserves as single IDs
   * (Sec. 4.5).  A leftmost-longest pass extracts them before
   * pre-tokenization, and the text between them is tokenized segment by
   * segment (no piece crosses a literal).  Literal i is
   * added_bytes[added_offsets[i] .. added_offsets[i+1]) (non-empty, strict
   * UTF-8, at most TT_MAX_ADDED_BYTES bytes, pairwise distinct) with ID
   * added_ids[i] (any non-negative value; it need not be in the vocabulary).
   * n_added == 0 means none. */
  int32_t n_added;
  const uint8_t* added_bytes;
  const int64_t* added_offsets; /* n_added + 1 entries, from 0, increasing */
  const int32_t* added_ids;
} tt_options;

#define TT_MAX_ADDED_BYTES 1024

/* tt_create with front-end options (opt may be NULL: no options).  All option
 * arrays are copied.  Handles with added tokens support tt_encode and
 * tt_encode_batch; the literal pass runs on the host before the request goes
 * to the device (as in the paper's service, Sec. 4.5), and the other entry
 * points return TT_ERR_BAD_ARG on such handles.  Invalid options return
 * TT_ERR_BAD_ARG (literals) or the codes of tt_create. */
int tt_create_ex(const tt_merge* merges, int32_t n_merges, const uint8_t* vocab_bytes,
                 const int64_t* vocab_offsets, int32_t vocab_size, int32_t pattern_id,
                 const tt_options* opt, tt_tokenizer** out);

/* Free the handle, its device tables and all its workspaces.  The caller must
 * not destroy a handle while a call on it is running.  NULL is ignored. */
void tt_destroy(tt_tokenizer* h);

/* ---- encode ---------------------------------------------------------- */
/* Tokenize one request held in host memory.
 *  utf8[len]      request bytes (host); len == 0 gives *out_len = 0.
 *  out_ids        host buffer of at least max(len, 1) IDs.
 *  out_len        receives the number of IDs written.
 * Blocks until out_ids/out_len are valid, with one host synchronisation for
 * requests up to 256 MiB (Sec. 4.3: the single-request path keeps the host
 * out of the chain).  The device reads the request straight from utf8 when
 * it is pinned host memory, else from a pinned copy, and writes the IDs
 * straight into out_ids when it is pinned host memory, else into pinned
 * staging that is then copied into out_ids.  When every ID of the handle's
 * vocabulary is below 65,536 (2^24), the staged IDs cross the bus in 2 (3)
 * bytes each and the copy into out_ids widens them (out_ids still receives
 * int32).
 * Staging copies of at least 256 KiB are split among the calling thread and
 * up to three worker threads of the library, which spin for 2 ms after a
 * copy, then sleep.  Longer requests take the length and the IDs back
 * in two copies.  NUL bytes are ordinary characters; no byte-order mark is
 * stripped.  Invalid UTF-8 returns TT_ERR_INVALID_UTF8 with *out_len = 0; the
 * contents of out_ids are then unspecified. */
int tt_encode(tt_tokenizer* h, const uint8_t* utf8, int64_t len, int32_t* out_ids,
              int64_t* out_len, void* stream);

/* Tokenize one request already resident in device memory; fully asynchronous.
 *  d_utf8[len]    request bytes (device), read-only, may be unaligned.
 *  d_out_ids      device buffer of at least max(len, 1) IDs.
 *  d_out_len      device int64_t: receives the number of IDs, or a negative
 *                 TT_ERR_* code if the device found an error (invalid UTF-8);
 *                 IDs are then unspecified.
 * Returns after enqueueing; host-detectable errors are returned directly. */
int tt_encode_device(tt_tokenizer* h, const uint8_t* d_utf8, int64_t len, int32_t* d_out_ids,
                     int64_t* d_out_len, void* stream);

/* tt_encode_device for callers that cannot allocate: code under stream
 * capture, tight serving loops, and hosts that forbid allocation while
 * serving.  The same arguments, layout, results and asynchrony as
 * tt_encode_device, and the same kernels; the call allocates nothing.  Its
 * workspace is one fixed array of device memory per GPU, reserved when the
 * library is loaded on that GPU and held until the process ends (about 43 MB
 * for TT_NOALLOC_MAX_BYTES); the call does no memory allocation, on the device
 * or on the host.
 *  - len > TT_NOALLOC_MAX_BYTES returns TT_ERR_TOO_LARGE (nothing is enqueued).
 *  - Handles with added-token literals return TT_ERR_BAD_ARG.
 *  - Every call on a GPU uses that GPU's one array: calls on one GPU whose
 *    work overlaps (other streams, other host threads, other handles) race and
 *    must be ordered by the caller.  Calls in stream order are independent:
 *    each call takes a new call number on the host, so the array's words from
 *    earlier calls are never mistaken for its own.  For the same reason a
 *    captured call cannot be replayed.
 *  - No stage events are recorded (tt_set_profiling does not apply). */
#define TT_NOALLOC_MAX_BYTES ((int64_t)1 << 21)
int tt_encode_device_noalloc(tt_tokenizer* h, const uint8_t* d_utf8, int64_t len, int32_t* d_out_ids,
                             int64_t* d_out_len, void* stream);

/* Tokenize a batch of independent documents in one call (Sec. 4.2: documents
 * are concatenated and runs are cut at document boundaries; no piece or token
 * crosses a document boundary).
 *  concat         all documents back to back (host), doc_offsets[n_docs] bytes.
 *  doc_offsets    n_docs+1 non-decreasing byte offsets, doc_offsets[0] == 0.
 *  out_ids        host buffer of at least max(doc_offsets[n_docs], 1) IDs.
 *  out_doc_offsets  n_docs+1 entries: document j's IDs are
 *                 out_ids[out_doc_offsets[j] .. out_doc_offsets[j+1]).
 * Every document must be valid UTF-8 on its own; otherwise
 * TT_ERR_INVALID_UTF8 and no output. */
int tt_encode_batch(tt_tokenizer* h, const uint8_t* concat, const int64_t* doc_offsets,
                    int32_t n_docs, int32_t* out_ids, int64_t* out_doc_offsets, void* stream);

/* ---- span export -------------------------------------------------------- */
/* Token IDs together with the source span of every token (Appendix, Route C:
 * span export; the records (id, a, b) of Definition d:records).  For
 * byte-level BPE a token's byte length is fixed by the vocabulary, so byte
 * offsets are a running sum of token lengths, and a running count of the
 * request's non-continuation bytes lifts them to character spans.  Span i is
 * four int32 values:
 *   [0] byte begin, [1] byte end      the token's bytes utf8[begin, end);
 *                                      the byte spans partition [0, len);
 *   [2] char begin, [3] char end      the characters (Unicode scalar values,
 *                                      counted from 0) that hold the token's
 *                                      first through last byte; tokens that
 *                                      split one multi-byte character all
 *                                      report that character.
 * Single requests only (no batches).
 *  utf8[len]      request bytes (host).
 *  out_ids        host buffer of at least max(len, 1) IDs.
 *  out_spans      host buffer of at least 4 * max(len, 1) int32 values.
 *  out_len        receives the number of IDs (and spans).
 * Blocks until the outputs are valid (two synchronisations; IDs and spans are
 * copied back together).  Invalid UTF-8 returns TT_ERR_INVALID_UTF8 and no
 * output.  The spans buffer of a stream's workspace is allocated on the first
 * call (16 bytes per byte of capacity). */
int tt_encode_spans(tt_tokenizer* h, const uint8_t* utf8, int64_t len, int32_t* out_ids, int32_t* out_spans,
                    int64_t* out_len, void* stream);

/* The same for a request already in device memory; fully asynchronous.
 *  d_utf8[len]    request bytes (device), read-only, may be unaligned.
 *  d_out_ids      device buffer of at least max(len, 1) IDs.
 *  d_out_spans    device buffer of at least 4 * max(len, 1) int32 values.
 *  d_out_len      device int64_t: the number of IDs, or a negative TT_ERR_*
 *                 code (invalid UTF-8), in which case IDs and spans are
 *                 unspecified. */
int tt_encode_spans_device(tt_tokenizer* h, const uint8_t* d_utf8, int64_t len, int32_t* d_out_ids,
                           int32_t* d_out_spans, int64_t* d_out_len, void* stream);

/* ---- split-level export (tests) ---------------------------------------- */
/* Pre-tokenization only: the UTF-8 byte offset of the first byte of every
 * piece, in order (Sec. 4.1: differential testing compares piece boundaries as
 * well as IDs, because an ID-level check can hide a split fault).
 *  utf8[len]          host bytes.
 *  out_piece_starts   host buffer of at least max(len, 1) entries.
 *  out_n              receives the number of pieces.
 * Invalid UTF-8 returns TT_ERR_INVALID_UTF8. */
int tt_pretokenize(tt_tokenizer* h, const uint8_t* utf8, int64_t len, int64_t* out_piece_starts,
                   int64_t* out_n, void* stream);

/* ---- incremental repair (stateful sessions) ------------------------------ */
/* A session holds the text of a growing request and the records (ID, byte
 * span, character span) of its full tokenization.  Appending text B to the
 * stored text A re-tokenizes only a window, the last w characters of A
 * followed by B, with this library, and splices the fresh records onto the
 * cached ones (Sec. 3.2, "Incremental repair"):
 *  - find the longest run of records on which cached and fresh tokenization
 *    agree in byte span and ID;
 *  - admit it only if it holds at least two tokens, covers more characters
 *    than the longest token of the vocabulary, and contains a synchronizing
 *    boundary (see tt_sync_boundaries) with its left neighbour inside the
 *    window (Appendix, Definition d:cert: such a boundary is a splice
 *    certificate, and Theorem t:main makes the splice exact);
 *  - keep the cached records up to the end of the run and the fresh records
 *    after it (Corollary c:shift: splicing at the end of the run equals
 *    splicing at the boundary inside it);
 *  - otherwise double w and try again, at most five times, then tokenize the
 *    whole text.
 * The resulting IDs are always identical to full tokenization of A ++ B; a
 * rejected window only costs more work.  Mid-text edits are not supported. */
typedef struct tt_session tt_session; /* opaque; not thread-safe */

/* Outcome of one append. */
typedef struct {
  int64_t kept;         /* leading tokens of the previous sequence kept as they were */
  int64_t n_tokens;     /* tokens of the whole text after the append             */
  int32_t windows;      /* windows tokenized (0 when the whole text was tokenized
                           directly: empty session, or a window reaching the
                           start of the text)                                    */
  int32_t full;         /* 1 if the whole text was tokenized                      */
  int64_t window_chars; /* width w of the window that was accepted (0 if full)  */
} tt_append_info;

/* New empty session on handle h.  window_chars is the first window width w in
 * characters (0 selects the paper's default, 512).  The session keeps a
 * pointer to h, which must outlive it; host memory grows with the text
 * (the bytes, 4 bytes per token ID and 16 bytes per token span). */
int tt_session_create(tt_tokenizer* h, int32_t window_chars, tt_session** out);

/* Free a session.  NULL is ignored. */
void tt_session_destroy(tt_session* s);

/* Append utf8[len] (host) to the session text and update its tokens.
 * The append must consist of whole characters: the text stays strict UTF-8,
 * else TT_ERR_INVALID_UTF8 and the session is unchanged.  The windows run on
 * `stream` (blocking calls of tt_encode_spans).  info (may be NULL) receives
 * the outcome; the new IDs are tokens [info.kept, info.n_tokens) of
 * tt_session_ids.  len == 0 changes nothing. */
int tt_session_append(tt_session* s, const uint8_t* utf8, int64_t len, tt_append_info* info, void* stream);

/* Copy tokens [from, from + count) of the session: IDs into out_ids (host,
 * count entries; may be NULL) and spans into out_spans (host, 4 * count
 * int32 values laid out as in tt_encode_spans; may be NULL).  The range must
 * lie inside [0, n_tokens), else TT_ERR_BAD_ARG. */
int tt_session_tokens(const tt_session* s, int64_t from, int64_t count, int32_t* out_ids, int32_t* out_spans);

/* Bytes, characters and tokens of the session text (any may be NULL). */
int tt_session_info(const tt_session* s, int64_t* n_bytes, int64_t* n_chars, int64_t* n_tokens);

/* Synchronizing boundaries of a text (host only; no GPU work, no handle):
 * out_mask[p] = 1 if byte position p (0 < p < len) lies between two
 * characters whose classes form a synchronizing transition of the pattern,
 * else 0.  At such a position every text that contains the two characters
 * there has a piece boundary, the pieces to its right do not depend on the
 * text before its left neighbour, and the pieces to its left do not depend on
 * the text after its right neighbour.  This is the certificate the paper's
 * splice check asks for (Appendix, "Discharging the certificate per family");
 * each pattern has its own set of such class pairs, derived here from its
 * alternatives.  Transitions, with O other,
 * L letter, N number, WS whitespace but CR/LF, NL CR/LF, SP U+0020, APO U+0027:
 *   GPT-2:   left and right classes differ, counting WS and NL as one class,
 *            and the left character is neither SP nor APO;
 *   cl100k:  (non-N, N); (N or NL, L); (L, N, NL or WS but SP, O);
 *            (L, N or O, WS); (L or N, NL).
 * Invalid UTF-8 next to a position gives 0 there.  out_mask has len entries
 * (host). */
int tt_sync_boundaries(int32_t pattern_id, const uint8_t* utf8, int64_t len, uint8_t* out_mask);

/* The splice decision of one window (host only; exported so that the
 * decision can be tested against records from any tokenizer).
 *  text[len]        the whole new text A ++ B (host).
 *  a_len            bytes of A; x  first byte of the window (a character
 *                   start, 0 < x < a_len).
 *  c_ids, c_spans   the n_c records of the tokenization of A (spans as in
 *                   tt_encode_spans, in text coordinates).
 *  f_ids, f_spans   the n_f records of the tokenization of text[x, len),
 *                   shifted to text coordinates (byte spans + x, character
 *                   spans + the characters before x).
 *  max_token_chars  the check's length bound (the longest token).
 * Returns 1 and sets *keep_c, *from_f when the window is admitted: the new
 * records are c[0, keep_c) followed by f[from_f, n_f).  Returns 0 when it is
 * rejected, or a negative TT_ERR_* code. */
int tt_splice_plan(int32_t pattern_id, const uint8_t* text, int64_t len, int64_t a_len, int64_t x,
                   const int32_t* c_ids, const int32_t* c_spans, int64_t n_c, const int32_t* f_ids,
                   const int32_t* f_spans, int64_t n_f, int64_t max_token_chars, int64_t* keep_c,
                   int64_t* from_f);

/* ---- misc ------------------------------------------------------------ */
/* Static English text for a status code. */
const char* tt_status_string(int status);

/* Number of merges and vocabulary size of a handle (for bindings). */
int tt_info(const tt_tokenizer* h, int32_t* n_merges, int32_t* vocab_size, int32_t* pattern_id);

/* ---- measurement ------------------------------------------------------- */
/* Stages of a call: one, the tile kernel (pre-tokenization, BPE and the
 * placement of every tile's outputs, Sec. 4.1-4.2), with the per-document
 * offsets of a batch. */
#define TT_N_STAGES 1

/* Record HIP events between the stages of every later call on this handle and
 * keep those of the most recent `n_calls` calls of each stream (0 stops
 * recording; at most 65,536).  For measurement only: each call then records
 * TT_N_STAGES + 1 events on its stream. */
int tt_set_profiling(tt_tokenizer* h, int32_t n_calls);

/* Elapsed milliseconds of the stages of the recorded calls on `stream`, oldest
 * call first, TT_N_STAGES entries per call.  Waits for those calls to finish.
 * out_ms holds `cap` entries; *n_out receives how many were written (whole
 * calls only; 0 if nothing was recorded). */
int tt_stage_times(tt_tokenizer* h, void* stream, double* out_ms, int32_t cap, int32_t* n_out);

#ifdef __cplusplus
}
#endif

#endif /* TOKTIER_H */
