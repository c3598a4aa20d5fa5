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
 * Character classes are those of the Oniguruma engine of HF tokenizers 0.22.2
 * (the paper pins class tables probed from the reference engine, Sec. 4.1). */
enum { TT_PATTERN_GPT2 = 0, TT_PATTERN_CL100K = 1 };

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
 *  pattern_id                TT_PATTERN_GPT2 or TT_PATTERN_CL100K.
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

/* Free the handle, its device tables and all its workspaces.  The caller must
 * not destroy a handle while a call on it is running.  NULL is ignored. */
void tt_destroy(tt_tokenizer* h);

/* ---- encode ---------------------------------------------------------- */
/* Tokenize one request held in host memory.
 *  utf8[len]      request bytes (host); len == 0 gives *out_len = 0.
 *  out_ids        host buffer of at least max(len, 1) IDs.
 *  out_len        receives the number of IDs written.
 * Blocks until out_ids/out_len are valid (two host synchronisations: one for
 * the device-side output length, one for the IDs).  NUL bytes are ordinary
 * characters; no byte-order mark is stripped.  Invalid UTF-8 returns
 * TT_ERR_INVALID_UTF8 and writes no IDs (*out_len = 0). */
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
