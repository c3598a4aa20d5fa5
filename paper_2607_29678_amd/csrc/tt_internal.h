// Internal definitions of the MI355X tokenizer library (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/toktier.h"
#include "tt_copy.h"

namespace tt {

// ---------------------------------------------------------------------------
// Character codes kept per byte in LDS by the tile kernel.
//   bits 0..2  class of the character whose first byte is here:
//              O other, L letter, N number, WS whitespace except CR/LF,
//              NL CR or LF, NONE for continuation bytes and positions
//              outside the text
//   bits 3..6  identity of a few characters the rules test by value
//   bit  7     a document starts here (no context crosses this position)
// ---------------------------------------------------------------------------
enum : uint32_t { C_O = 0, C_L = 1, C_N = 2, C_WS = 3, C_NL = 4, C_NONE = 7 };
enum : uint32_t {
  I_NONE = 0,
  I_SP = 1,   // U+0020
  I_APO = 2,  // U+0027
  I_S = 3,    // contraction letters, folded per pattern
  I_T = 4,
  I_R = 5,
  I_E = 6,
  I_V = 7,
  I_M = 8,
  I_L = 9,
  I_D = 10
};
constexpr uint32_t CODE_DOCSTART = 0x80u;
__host__ __device__ inline uint32_t code_cls(uint32_t c) { return c & 7u; }
__host__ __device__ inline uint32_t code_id(uint32_t c) { return (c >> 3) & 15u; }

// ---------------------------------------------------------------------------
// Token IDs inside the library.  Byte b is ID b and the result of the merge
// of rank r is ID 256 + r; the output stage maps them to the caller's IDs.
// A proper merge list makes this a bijection onto the IDs BPE can produce
// (every operand is a byte or an earlier result, and results are unique), and
// it lets a merge table slot hold the key and the rank in 64 bits: the result
// of a merge is implied by its rank.
// ---------------------------------------------------------------------------
constexpr uint32_t ID_BITS = 21;
constexpr uint32_t ID_LIMIT = (1u << ID_BITS) - 1u;       // internal IDs are < ID_LIMIT
constexpr uint32_t MAX_MERGES = ID_LIMIT - 256u;          // 2,096,895
constexpr uint64_t KEY_MASK = (1ull << (2 * ID_BITS)) - 1ull;
constexpr uint64_t SLOT_EMPTY = ~0ull;                    // its key is (ID_LIMIT, ID_LIMIT)
constexpr uint32_t RANK_INF = 0xFFFFFFFFu;

__host__ __device__ inline uint64_t slot_key(uint32_t a, uint32_t b) {
  return (uint64_t)a | ((uint64_t)b << ID_BITS);
}

// A value that is the same in every lane of the wave, moved to a scalar
// register (values read from LDS otherwise occupy a vector register per lane).
__device__ __forceinline__ uint32_t wave_uniform(uint32_t x) {
  return (uint32_t)__builtin_amdgcn_readfirstlane((int)x);
}

// Bucket of a 32-bit hash among nb buckets: the high word of hash * nb (any
// bucket count; the high bits of a multiplicative hash are the good ones).
__host__ __device__ inline uint32_t bucket_of(uint32_t h, uint32_t nb) { return (uint32_t)(((uint64_t)h * nb) >> 32); }

// Two bucket hashes of a pair (multiplicative).
__host__ __device__ inline uint32_t pair_hash(uint32_t a, uint32_t b) { return (a * 0x9E3779B1u + b) * 0x85EBCA77u; }
__host__ __device__ inline uint32_t pair_hash2(uint32_t a, uint32_t b) {
  return ((b * 0xC2B2AE3Du) ^ (a + 0x165667B1u)) * 0x27D4EB2Fu;
}

// The merge table is a two-choice cuckoo table of 16-byte buckets holding
// two slots each: a pair lives in one of the two buckets its hashes name, so
// every lookup is exactly two independent 16-byte loads (one memory round
// trip, no probe chain).  Pairs of two bytes, the only pairs before any
// merge, also have a direct 64 K-entry rank table.
typedef uint64_t u64x2 __attribute__((ext_vector_type(2)));

struct ProbeIssued {
  u64x2 x, y;
};
__device__ __forceinline__ ProbeIssued probe_issue(const u64x2* __restrict__ tab, uint32_t nb, uint32_t a,
                                                   uint32_t b) {
  return ProbeIssued{tab[bucket_of(pair_hash(a, b), nb)], tab[bucket_of(pair_hash2(a, b), nb)]};
}
// Only the high word of the matching slot is kept (key bits 32..41 below the
// rank): no empty slot matches, because no internal ID has all 21 bits set.
__device__ __forceinline__ uint32_t probe_finish(const ProbeIssued& p, uint32_t a, uint32_t b) {
  const uint32_t klo = a | (b << ID_BITS), khi = b >> (32 - ID_BITS);
  constexpr uint32_t HI_KEY = (1u << (2 * ID_BITS - 32)) - 1u;
  uint32_t hi = 0xFFFFFFFFu;
  auto check = [&](uint64_t v) {
    const uint32_t vh = (uint32_t)(v >> 32);
    hi = ((uint32_t)v == klo && (vh & HI_KEY) == khi) ? vh : hi;
  };
  check(p.x.x);
  check(p.x.y);
  check(p.y.x);
  check(p.y.y);
  return hi == 0xFFFFFFFFu ? RANK_INF : hi >> (2 * ID_BITS - 32);
}
// Rank of the pair (a, b), or RANK_INF if no merge joins it.
__device__ __forceinline__ uint32_t probe_rank(const u64x2* __restrict__ tab, uint32_t nb, uint32_t a,
                                               uint32_t b) {
  return probe_finish(probe_issue(tab, nb, a, b), a, b);
}

// Whole-unit dictionary: a unit of 3..DICT_MAX bytes whose BPE is a single
// token is found with one lookup.  An entry holds the unit's bytes (zero
// padded, little-endian words), and its length and token: (id << 4) | length.
// Two-choice cuckoo table of two entries per bucket; a unit lives in one of
// the two buckets its hashes name (four 16-byte loads, one round trip).
constexpr int DICT_MAX = 12;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__host__ __device__ inline uint32_t unit_hash(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t len) {
  uint32_t x = w0 * 0x9E3779B1u + w1 * 0x85EBCA77u + w2 * 0xC2B2AE3Du + len;
  x ^= x >> 15;
  return x * 0x2C1B3C6Du;
}
__host__ __device__ inline uint32_t unit_hash2(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t len) {
  uint32_t x = (w0 * 0x27D4EB2Fu) ^ (w1 * 0x165667B1u) ^ (w2 * 0xD3A2646Cu) ^ (len * 0xFD7046C5u);
  x ^= x >> 13;
  return x * 0x297A2D39u;
}
constexpr uint32_t DICT_NONE = 0xFFFFFFFFu;
__device__ __forceinline__ bool dict_match(const u32x4& e, uint32_t w0, uint32_t w1, uint32_t w2, uint32_t len) {
  return e.x == w0 && e.y == w1 && e.z == w2 && (e.w & 15u) == len;
}
__device__ __forceinline__ uint32_t dict_find(const u32x4* __restrict__ dict, uint32_t nb, uint32_t w0, uint32_t w1,
                                              uint32_t w2, uint32_t len) {
  const uint32_t b1 = 2u * bucket_of(unit_hash(w0, w1, w2, len), nb);
  const uint32_t b2 = 2u * bucket_of(unit_hash2(w0, w1, w2, len), nb);
  const u32x4 e0 = dict[b1], e1 = dict[b1 + 1], e2 = dict[b2], e3 = dict[b2 + 1];
  uint32_t r = DICT_NONE;
  r = dict_match(e0, w0, w1, w2, len) ? e0.w >> 4 : r;
  r = dict_match(e1, w0, w1, w2, len) ? e1.w >> 4 : r;
  r = dict_match(e2, w0, w1, w2, len) ? e2.w >> 4 : r;
  r = dict_match(e3, w0, w1, w2, len) ? e3.w >> 4 : r;
  return r;
}

// Long-unit dictionary: the same for units of DICT_MAX+1..DICT2_MAX bytes.
// An entry is two 16-byte words, {bytes 0..15} and {bytes 16..23, (id << 5) |
// length, 0}; one entry per bucket, two choices (four 16-byte loads).
constexpr int DICT2_MAX = 24;

__host__ __device__ inline uint32_t unit_hash6(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3, uint32_t w4,
                                               uint32_t w5, uint32_t len) {
  uint32_t x = w0 * 0x9E3779B1u + w1 * 0x85EBCA77u + w2 * 0xC2B2AE3Du + w3 * 0x27D4EB2Fu + w4 * 0x165667B1u +
               w5 * 0xD3A2646Cu + len;
  x ^= x >> 15;
  return x * 0x2C1B3C6Du;
}
__host__ __device__ inline uint32_t unit_hash6b(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3, uint32_t w4,
                                                uint32_t w5, uint32_t len) {
  uint32_t x = (w0 * 0x27D4EB2Fu) ^ (w1 * 0x165667B1u) ^ (w2 * 0xD3A2646Cu) ^ (w3 * 0xFD7046C5u) ^
               (w4 * 0xB55A4F09u) ^ (w5 * 0x9E3779B1u) ^ (len * 0x85EBCA77u);
  x ^= x >> 13;
  return x * 0x297A2D39u;
}
__device__ __forceinline__ uint32_t dict2_find(const u32x4* __restrict__ dict, uint32_t nb, const uint32_t (&w)[6],
                                               uint32_t len) {
  const uint32_t b1 = 2u * bucket_of(unit_hash6(w[0], w[1], w[2], w[3], w[4], w[5], len), nb);
  const uint32_t b2 = 2u * bucket_of(unit_hash6b(w[0], w[1], w[2], w[3], w[4], w[5], len), nb);
  const u32x4 a0 = dict[b1], a1 = dict[b1 + 1], c0 = dict[b2], c1 = dict[b2 + 1];
  uint32_t r = DICT_NONE;
  if (a0.x == w[0] && a0.y == w[1] && a0.z == w[2] && a0.w == w[3] && a1.x == w[4] && a1.y == w[5] &&
      (a1.z & 31u) == len)
    r = a1.z >> 5;
  if (c0.x == w[0] && c0.y == w[1] && c0.z == w[2] && c0.w == w[3] && c1.x == w[4] && c1.y == w[5] &&
      (c1.z & 31u) == len)
    r = c1.z >> 5;
  return r;
}

// Vocabulary strings longer than DICT2_MAX (piece probes under
// ignore_merges): one 16-byte entry {hash, length, ID, offset of the bytes in
// a blob} per bucket slot, two slots per bucket, two choices from two hashes
// of the bytes; a hit on (hash, length) is confirmed by comparing the bytes.
__host__ __device__ inline uint32_t long_hash_step(uint32_t h, uint32_t b) { return (h ^ b) * 0x01000193u; }
constexpr uint32_t LONG_SEED1 = 0x811C9DC5u, LONG_SEED2 = 0x9747B28Cu;
__host__ __device__ inline uint32_t long_hash_final(uint32_t h, uint32_t len) {
  h ^= len * 0x9E3779B1u;
  h ^= h >> 16;
  h *= 0x85EBCA6Bu;
  h ^= h >> 13;
  return h;
}

// Everything a kernel needs to know about a tokenizer handle.
struct DevTables {
  const u64x2* slots;       // cuckoo buckets of two slots: key (left | right << 21), rank in bits 42..63
  uint32_t nb;              // bucket count
  const uint32_t* pair0;    // [65536] rank of the byte pair (x << 8 | y), or RANK_INF
  const uint32_t* join;     // [2048] bit (x << 8 | y): some merge joins a token ending
                            // in byte x to a token starting with byte y
  const int32_t* ext_id;    // [n_ids] caller's ID of every internal ID
  uint32_t n_ids;           // 256 + M
  const u32x4* dict;        // whole-unit dictionary (two entries per bucket)
  uint32_t dnb;             // dictionary bucket count
  const u32x4* dict2;       // long-unit dictionary (one two-word entry per bucket)
  uint32_t dnb2;            // its bucket count
  const uint32_t* tok_len;  // [n_ids] byte length of every internal ID (span export)
  // ignore_merges: whole-piece probes of every vocabulary string (lowest ID)
  uint32_t vmax;            // longest vocabulary string in bytes (0: no probes)
  const u32x4* vdict;       // strings of 2..DICT_MAX bytes, whole-unit dictionary layout
  uint32_t vdnb;
  const u32x4* vdict2;      // strings of DICT_MAX+1..DICT2_MAX bytes, long-unit dictionary layout
  uint32_t vdnb2;
  const u32x4* vlong;       // longer strings: {hash, length, ID, blob offset}, two per bucket
  uint32_t vlnb;
  const uint8_t* vblob;     // bytes of the longer strings
};

// ---------------------------------------------------------------------------
// Control words of a workspace.  Nothing is cleared between calls: every call
// has an epoch (1, 2, ...), words that later blocks wait on carry the epoch of
// the call that wrote them, and the tile ticket only ever grows (a call's
// tiles are tickets [ticket_base, ticket_base + n_tiles)).
// ---------------------------------------------------------------------------
struct Ctrl {
  uint32_t tile_ticket;
  uint32_t pad;
};
constexpr uint32_t EPOCH_LIMIT = 0x7FFFFFFFu;  // epochs are 1 .. EPOCH_LIMIT - 1 (31 bits)

constexpr uint32_t NO_START = 0xFFFFFFFFu;  // tile_last: no unit starts in the tile

// Buffers and parameters of one call (all device memory).
struct Work {
  const uint8_t* text;      // request bytes (caller's or staged)
  uint32_t n;               // bytes
  const int64_t* doc_off;   // batch: n_docs+1 byte offsets, else nullptr
  int32_t n_docs;
  Ctrl* ctrl;
  uint32_t epoch;           // this call's epoch
  uint32_t ticket_base;     // first tile ticket of this call
  uint32_t n_tiles;
  uint64_t* tile_sum;       // [tiles] (epoch << 32) | trailing-run summary (cl100k carries), or the
                            // start of the tile's last piece (walked patterns)
  uint64_t* tile_end;       // [tiles] walked patterns: (epoch << 32) | end of the tile's last piece
  uint64_t* tile_last;      // [tiles] (epoch << 32) | last unit start in the tile, or NO_START
  uint64_t* tile_agg;       // [tiles] output counts for the placement look-back (epoch-tagged)
  uint64_t* tile_cagg;      // [tiles] span export: non-continuation byte counts, same protocol
  uint32_t* tile_pre;       // batch: [tiles] outputs of all earlier tiles
  uint32_t* stage;          // [n] tokens of incoming units, at the unit's first byte
  uint32_t* unit_tile;      // batch: [n] processing tile of the unit starting at a byte
  uint32_t* unit_pos;       // batch: [n] its first output within that tile's outputs
  uint32_t* scratch;        // rows of units longer than 64 bytes: 4 * n words, then n / 16 + 8 masks
  uint32_t* ccount;         // span export: [n/4 + 1] non-continuation bytes before byte 4w
  int32_t* out_spans;       // span export: [T][4] byte begin, byte end, char begin, char end
  int32_t* out_ids;         // output (caller IDs, or piece offsets for the split export)
  uint16_t* out16;          // encode without span export: when set, the IDs go here as 16-bit
                            // values instead (their low 16 bits when out_hi is set too)
  uint8_t* out_hi;          // with out16: bits 16..23 of every ID (every caller ID is below 2^24)
  int64_t* out_len;         // output length, or -error
  int64_t* out_doc_off;     // batch: n_docs+1 output offsets (device)
};

// Tiles and geometry --------------------------------------------------------
constexpr int PT_THREADS = 512;                   // tile block
constexpr int PT_BPT = 4;                          // bytes per thread
constexpr int PT_WIN = PT_THREADS * PT_BPT;        // window bytes in LDS
constexpr int PT_HALO = 32;                        // context bytes each side
constexpr int PT_OWN = PT_WIN - 2 * PT_HALO;       // bytes a tile decides
constexpr int PT_PAD = 8;  // LDS arrays also hold window positions [-8, 0) and [PT_WIN, PT_WIN + 16)

constexpr int SMALL_MAX = 16;                      // thread-per-unit limit (bytes)
constexpr int TH_THREADS = 256;                    // threads of a tile that run the thread engine
constexpr int WAVE_MAX = 128;                      // wave-per-unit limit (bytes)
constexpr int ROWS_LDS = 480;                      // longer units: rows in LDS up to this length

inline uint32_t n_tiles_for(uint32_t n) { return (n + PT_OWN - 1) / PT_OWN; }

// Launchers (defined in the .hip files) -------------------------------------
// mode 0: split export (outputs are piece byte offsets); mode 1: encode;
// mode 2: encode with span export (single requests)
// ignore: probe whole pieces in the vocabulary first (modes 1 and 2)
hipError_t launch_tile(const Work& w, const DevTables& t, int pattern, int mode, bool ignore, hipStream_t s);
hipError_t launch_doc_offsets(const Work& w, hipStream_t s);
// span export, after the tile kernel: byte ends and character spans
hipError_t launch_spans(const Work& w, hipStream_t s);

// Facts of a handle for the host-side session code and the entry points
// outside tt_api.hip.
int handle_pattern(const tt_tokenizer* h);
int handle_device(const tt_tokenizer* h);
bool handle_ignore(const tt_tokenizer* h);  // ignore_merges
DevTables handle_tables(const tt_tokenizer* h);
bool handle_has_added(const tt_tokenizer* h);  // added-token literals (sessions do not take them)
uint32_t handle_max_token_bytes(const tt_tokenizer* h);  // longest token, in bytes
// span export of a small host request with one synchronisation (pinned buffers)
int encode_spans_pinned(tt_tokenizer* h, const uint8_t* h_in, int64_t len, int32_t* h_ids, int32_t* h_spans,
                        int64_t* h_len, void* stream);

}  // namespace tt
