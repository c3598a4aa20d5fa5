// Internal definitions of the MI355X tokenizer library (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/toktier.h"

namespace tt {

// ---------------------------------------------------------------------------
// Character codes kept per byte in LDS by the pre-tokenization kernel.
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

// Device control block of one call.  Zeroed by the first kernel of the chain.
struct Ctrl {
  uint32_t tile_ticket;   // pre-tokenization tiles taken
  uint32_t n_pieces;      // P, written by the last pre-tokenization tile
  uint32_t error;         // 0, or the magnitude of a TT_ERR_* code
  uint32_t n_long;        // pieces queued for the wave engine
  uint32_t long_ticket;   // wave-engine queue head
  uint32_t n_big;         // pieces queued for the block engine
  uint32_t big_ticket;    // block-engine queue head
  uint32_t ctile_ticket;  // compaction tiles taken
  uint32_t small_done;    // (unused; keeps the struct 8-byte aligned)
  uint32_t pad;
  int64_t out_len;        // T, written by the last compaction tile
};

// One slot of the open-addressing merge table: key (left, right), value
// (rank, result).  Empty slots have left == EMPTY.
struct MergeSlot {
  uint32_t left, right, rank, result;
};
constexpr uint32_t EMPTY = 0xFFFFFFFFu;
constexpr uint32_t RANK_INF = 0xFFFFFFFFu;

__host__ __device__ inline uint32_t pair_hash(uint32_t a, uint32_t b) {
  uint32_t h = a * 0x9E3779B1u ^ (b + 0x7F4A7C15u) * 0x85EBCA77u;
  h ^= h >> 15;
  h *= 0x2C1B3C6Du;
  h ^= h >> 12;
  h *= 0x297A2D39u;
  h ^= h >> 15;
  return h;
}

// Slot index where the search for the pair (a, b) starts.
__device__ __forceinline__ uint32_t probe_start(uint32_t mask, uint32_t a, uint32_t b) {
  return pair_hash(a, b) & mask;
}

// One 16-byte slot, fetched with a single 128-bit load.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 load_slot(const MergeSlot* __restrict__ tab, uint32_t i) {
  u32x4 v = reinterpret_cast<const u32x4*>(tab)[i];
  return make_uint4(v.x, v.y, v.z, v.w);
}

// Finish a probe whose first slot `s` (at index i) is already loaded: rank
// and result of the pair (a, b), or RANK_INF if the pair has no merge.
__device__ __forceinline__ uint2 probe_finish(const MergeSlot* __restrict__ tab, uint32_t mask, uint32_t i,
                                              uint4 s, uint32_t a, uint32_t b) {
  while (!((s.x == a) & (s.y == b)) && s.x != EMPTY) {
    i = (i + 1) & mask;
    s = load_slot(tab, i);
  }
  return (s.x == a) & (s.y == b) ? make_uint2(s.z, s.w) : make_uint2(RANK_INF, 0u);
}

__device__ __forceinline__ uint2 probe_pair(const MergeSlot* __restrict__ tab, uint32_t mask, uint32_t a,
                                           uint32_t b) {
  uint32_t i = probe_start(mask, a, b);
  return probe_finish(tab, mask, i, load_slot(tab, i), a, b);
}

// Everything a kernel needs to know about a tokenizer handle.
struct DevTables {
  const MergeSlot* slots;  // open-addressing merge table
  uint32_t mask;           // slot count - 1
  const int32_t* byte_id;  // [256] base ID of each byte
};

// Buffers of one call (all device memory).
struct Work {
  const uint8_t* text;      // request bytes (caller's or staged)
  uint32_t n;               // bytes
  const int64_t* doc_off;   // batch: n_docs+1 byte offsets, else nullptr
  int32_t n_docs;
  Ctrl* ctrl;
  // "pieces" below are the units of the call: pre-tokenization pieces for the
  // split-level export, BPE segments of pieces for encoding
  uint32_t* piece_off;      // [P+1] byte offset of each unit start, then n
  uint32_t* piece_cnt;      // [P] tokens per unit
  uint32_t* piece_out;      // [P+1] output offset of each unit
  int32_t* ids;             // [n] per-piece IDs stored at the piece's byte offset
  uint32_t* long_list;      // [P] pieces for the wave engine
  uint32_t* big_list;       // [P] pieces for the block engine
  uint64_t* tile_status;    // pre-tokenization look-back words
  uint32_t* tile_summary;   // pre-tokenization run summaries (cl100k carries)
  uint64_t* ctile_status;   // compaction look-back words
  uint32_t* scratch32;      // [6 * n] block-engine double buffers
  int32_t* out_ids;         // output IDs
  int64_t* out_len;         // output length (or -error)
  int64_t* out_doc_off;     // batch: n_docs+1 output offsets (device)
};

// Tiles and geometry --------------------------------------------------------
constexpr int PT_THREADS = 1024;                  // pre-tokenization block
constexpr int PT_BPT = 2;                          // bytes per thread
constexpr int PT_WIN = PT_THREADS * PT_BPT;        // window bytes in LDS
constexpr int PT_HALO = 32;                        // context bytes each side
constexpr int PT_OWN = PT_WIN - 2 * PT_HALO;       // bytes a tile decides

constexpr int SMALL_MAX = 16;                      // thread-per-piece limit (bytes)
constexpr int WAVE_MAX = 512;                      // wave engine limit (bytes)
constexpr int CT_THREADS = 256;                    // compaction block
constexpr int CT_PPT = 8;                          // pieces per thread
constexpr int CT_TILE = CT_THREADS * CT_PPT;

inline uint32_t pt_tiles(uint32_t n) { return (n + PT_OWN - 1) / PT_OWN; }
inline uint32_t ct_tiles_cap(uint32_t n) { return (n + CT_TILE - 1) / CT_TILE + 1; }

// Launchers (defined in the .hip files) -------------------------------------
hipError_t launch_reset(const Work& w, uint32_t n_pt_tiles, uint32_t n_ct_tiles, hipStream_t s);
hipError_t launch_pretok(const Work& w, int pattern, uint32_t n_pt_tiles, const uint32_t* join_bits, bool seg,
                         hipStream_t s);
hipError_t launch_bpe_small(const Work& w, const DevTables& t, hipStream_t s);
hipError_t launch_bpe_wave(const Work& w, const DevTables& t, hipStream_t s);
hipError_t launch_bpe_block(const Work& w, const DevTables& t, hipStream_t s);
hipError_t launch_compact(const Work& w, uint32_t n_ct_tiles, hipStream_t s);
hipError_t launch_doc_offsets(const Work& w, hipStream_t s);

}  // namespace tt
