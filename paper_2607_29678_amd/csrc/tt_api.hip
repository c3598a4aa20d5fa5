// C ABI of the tokenizer: handle creation and validation, per-stream
// workspaces, and the launch chain of one call.
//
// Chain of one request (all on the caller's stream, no host round trip
// between kernels; Sec. 4.3 keeps piece counts, dispatch lists and the output
// length on the device and sizes launches from buffer capacity):
//   tile kernel (pre-tokenize + BPE + placement of every tile's outputs)
//   [-> document offsets, for batches]
// The host synchronises twice per blocking call: once for the output length,
// once for the IDs.
#include <algorithm>
#include <cstdint>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <unordered_map>
#include <unordered_set>
#include <vector>

#include "tt_internal.h"

using namespace tt;

namespace {

// Stages of one call, in launch order (profiling names them in this order).
enum { ST_TILE, N_STAGES };

struct Workspace {
  uint64_t cap = 0;           // bytes of request this workspace holds
  int64_t doc_cap = 0;        // documents the batch buffers hold
  void* dmem = nullptr;       // one device allocation for everything below
  Work w{};                   // device pointers (text/out set per call)
  uint32_t epoch = 0;         // epoch of the latest call
  uint32_t ticket_base = 0;   // first tile ticket of the next call
  size_t ctl_bytes = 0;       // control block and tile words, cleared when allocated
  uint8_t* d_in = nullptr;    // staged request bytes (host calls)
  int32_t* d_out = nullptr;   // IDs (host calls)
  int64_t* d_len = nullptr;   // output length (host calls)
  int64_t* d_docs = nullptr;  // batch: document byte offsets
  int64_t* d_out_docs = nullptr;
  int32_t* d_spans = nullptr;  // span export (host calls): [span_cap][4], allocated on first use
  uint64_t span_cap = 0;
  int64_t* h_len = nullptr;   // pinned readback word
  // tt_encode: pinned staging, sized with the capacity
  uint64_t pin_cap = 0;        // bytes of request it holds
  uint8_t* h_in = nullptr;     // request bytes for the DMA (pageable callers)
  int32_t* h_ids = nullptr;    // IDs from the device (pageable callers)
  // profiling: stage boundaries of the most recent calls, a ring of
  // `ring` calls with N_STAGES + 1 events each
  std::vector<hipEvent_t> ev;
  int ring = 0;          // calls the ring holds
  int64_t n_calls = 0;   // calls recorded since profiling was enabled
};

// Strict UTF-8 validation on the host (added-token literals).
bool valid_utf8(const uint8_t* t, int64_t n) {
  int64_t i = 0;
  while (i < n) {
    const uint32_t b0 = t[i];
    const int len = b0 < 0x80u ? 1 : b0 < 0xC2u ? 0 : b0 < 0xE0u ? 2 : b0 < 0xF0u ? 3 : b0 < 0xF5u ? 4 : 0;
    if (len == 0 || i + len > n) return false;
    if (len > 1) {
      const uint32_t b1 = t[i + 1];
      const uint32_t lo = b0 == 0xE0u ? 0xA0u : b0 == 0xF0u ? 0x90u : 0x80u;
      const uint32_t hi = b0 == 0xEDu ? 0x9Fu : b0 == 0xF4u ? 0x8Fu : 0xBFu;
      if (b1 < lo || b1 > hi) return false;
      for (int k = 2; k < len; ++k)
        if ((t[i + k] & 0xC0u) != 0x80u) return false;
    }
    i += len;
  }
  return true;
}

// Added-token literals and their leftmost-longest extraction (Sec. 4.5: a
// leftmost-longest literal pass runs before the tokenizer family handles the
// remaining segments).  Candidates are found per distinct first byte with
// memchr, the longest literal at each candidate position is kept, and the
// scan takes every candidate that starts at or after the end of the last
// literal taken.
struct AddedSet {
  std::vector<std::string> lits;
  std::vector<int32_t> ids;
  std::vector<std::vector<uint32_t>> by_first;  // [256] literal indices, longest first
  std::vector<uint8_t> firsts;                  // distinct first bytes
  struct Match {
    int64_t s, e;
    int32_t id;
  };

  bool empty() const { return lits.empty(); }
  void add(const std::string& lit, int32_t id) {
    lits.push_back(lit);
    ids.push_back(id);
  }
  void finish() {
    by_first.assign(256, {});
    for (uint32_t i = 0; i < lits.size(); ++i) by_first[(uint8_t)lits[i][0]].push_back(i);
    firsts.clear();
    for (int b = 0; b < 256; ++b) {
      auto& v = by_first[b];
      if (v.empty()) continue;
      firsts.push_back((uint8_t)b);
      std::stable_sort(v.begin(), v.end(), [&](uint32_t x, uint32_t y) { return lits[x].size() > lits[y].size(); });
    }
  }
  // the longest literal starting at t[p] (first byte already known to match)
  bool longest_at(const uint8_t* t, int64_t n, int64_t p, Match& m) const {
    for (uint32_t i : by_first[t[p]]) {
      const std::string& l = lits[i];
      if ((int64_t)l.size() <= n - p && std::memcmp(t + p, l.data(), l.size()) == 0) {
        m = Match{p, p + (int64_t)l.size(), ids[i]};
        return true;
      }
    }
    return false;
  }
  void extract(const uint8_t* t, int64_t n, std::vector<Match>& out) const {
    out.clear();
    std::vector<Match> cand;
    Match m;
    if (firsts.size() <= 4) {
      for (uint8_t b : firsts) {
        const uint8_t* q = t;
        while ((q = static_cast<const uint8_t*>(std::memchr(q, b, (size_t)(t + n - q)))) != nullptr) {
          if (longest_at(t, n, q - t, m)) cand.push_back(m);
          ++q;
        }
      }
      if (firsts.size() > 1)
        std::sort(cand.begin(), cand.end(), [](const Match& x, const Match& y) { return x.s < y.s; });
    } else {
      for (int64_t p = 0; p < n; ++p)
        if (!by_first[t[p]].empty() && longest_at(t, n, p, m)) cand.push_back(m);
    }
    int64_t covered = 0;
    for (const Match& c : cand)
      if (c.s >= covered) {
        out.push_back(c);
        covered = c.e;
      }
  }
};

}  // namespace

struct tt_tokenizer {
  int pattern = 0;
  int32_t n_merges = 0;
  int32_t vocab_size = 0;
  int device = 0;
  int profile = 0;  // calls whose stage events are kept (0: no events)
  u64x2* d_slots = nullptr;    // cuckoo buckets
  uint32_t nb = 0;             // merge-table buckets
  uint32_t* d_pair0 = nullptr;  // [65536] byte-pair ranks
  u32x4* d_dict = nullptr;      // whole-unit dictionary
  uint32_t dnb = 0;             // dictionary buckets
  u32x4* d_dict2 = nullptr;     // long-unit dictionary
  uint32_t dnb2 = 0;            // its buckets
  int32_t* d_ext = nullptr;    // [256 + M] caller's ID of every internal ID
  uint32_t* d_toklen = nullptr;  // [256 + M] byte length of every internal ID
  uint32_t n_ids = 0;
  int id_bits = 32;            // 16 or 24 when every caller ID fits: staged IDs cross the bus in that many bits
  uint32_t max_tok_bytes = 1;  // byte length of the longest token (incremental repair)
  bool ignore = false;         // ignore_merges: whole pieces probed in the vocabulary first
  uint32_t vmax = 0;           // longest vocabulary string (bytes) of the probes
  u32x4* d_vdict = nullptr;    // probe tables (see DevTables)
  uint32_t vdnb = 0;
  u32x4* d_vdict2 = nullptr;
  uint32_t vdnb2 = 0;
  u32x4* d_vlong = nullptr;
  uint32_t vlnb = 0;
  uint8_t* d_vblob = nullptr;
  AddedSet added;              // added-token literals (host-side extraction)
  uint32_t* d_join = nullptr;  // [2048] bit (x << 8 | y) set if some merge joins a token ending in
                               // byte x to a token starting with byte y
  std::mutex mu;
  std::unordered_map<hipStream_t, Workspace*> ws;
};

namespace {

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

void free_ws(Workspace* s) {
  if (!s) return;
  if (s->dmem) (void)hipFree(s->dmem);
  if (s->d_docs) (void)hipFree(s->d_docs);
  if (s->d_spans) (void)hipFree(s->d_spans);
  if (s->h_len) (void)hipHostFree(s->h_len);
  if (s->h_in) (void)hipHostFree(s->h_in);
  if (s->h_ids) (void)hipHostFree(s->h_ids);
  for (auto e : s->ev)
    if (e) (void)hipEventDestroy(e);
  delete s;
}

// (Re)allocate the device buffers of a workspace for requests up to `need` bytes.
int ws_reserve(Workspace* s, uint64_t need, hipStream_t st) {
  if (need <= s->cap) return TT_OK;
  // earlier asynchronous calls on this stream may still use the old buffers
  if (s->dmem && hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
  // grow to a power of two, so that requests of about the same size share one
  // allocation (a reallocation synchronises the stream)
  uint64_t cap = 65536;
  while (cap < need || cap < s->cap * 2) cap <<= 1;
  if (cap > (uint64_t)TT_MAX_BYTES) cap = std::max<uint64_t>(need, (uint64_t)TT_MAX_BYTES);
  if (s->dmem) {
    (void)hipFree(s->dmem);
    s->dmem = nullptr;
    s->cap = 0;
  }
  const uint64_t N = cap;
  const uint64_t NT = n_tiles_for((uint32_t)N) + 1;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  // words that carry epochs or the ticket come first: they are cleared once here
  size_t o_ctrl = take(sizeof(Ctrl));
  size_t o_tsum = take(8 * NT);
  size_t o_tend = take(8 * NT);
  size_t o_tlast = take(8 * NT);
  size_t o_tagg = take(8 * NT);
  size_t o_tcagg = take(8 * NT);
  const size_t ctl_bytes = off;
  size_t o_tpre = take(4 * NT);
  size_t o_stage = take(4 * N);
  size_t o_utile = take(4 * N);
  size_t o_upos = take(4 * N);
  size_t o_scr = take(4 * 4 * N + 8 * (N / 16 + 8));
  size_t o_ccount = take(4 * (N / 4 + 2));
  size_t o_in = take(N + 64);
  size_t o_out = take(4 * N);
  size_t o_len = take(8);
  void* mem = nullptr;
  if (hipMalloc(&mem, off) != hipSuccess) return TT_ERR_OOM;
  if (hipMemsetAsync(mem, 0, ctl_bytes, st) != hipSuccess) {
    (void)hipFree(mem);
    return TT_ERR_HIP;
  }
  uint8_t* b = static_cast<uint8_t*>(mem);
  s->dmem = mem;
  s->cap = cap;
  s->ctl_bytes = ctl_bytes;
  s->epoch = 0;
  s->ticket_base = 0;
  Work& w = s->w;
  w.ctrl = reinterpret_cast<Ctrl*>(b + o_ctrl);
  w.tile_sum = reinterpret_cast<uint64_t*>(b + o_tsum);
  w.tile_end = reinterpret_cast<uint64_t*>(b + o_tend);
  w.tile_last = reinterpret_cast<uint64_t*>(b + o_tlast);
  w.tile_agg = reinterpret_cast<uint64_t*>(b + o_tagg);
  w.tile_cagg = reinterpret_cast<uint64_t*>(b + o_tcagg);
  w.ccount = reinterpret_cast<uint32_t*>(b + o_ccount);
  w.tile_pre = reinterpret_cast<uint32_t*>(b + o_tpre);
  w.stage = reinterpret_cast<uint32_t*>(b + o_stage);
  w.unit_tile = reinterpret_cast<uint32_t*>(b + o_utile);
  w.unit_pos = reinterpret_cast<uint32_t*>(b + o_upos);
  w.scratch = reinterpret_cast<uint32_t*>(b + o_scr);
  s->d_in = b + o_in;
  s->d_out = reinterpret_cast<int32_t*>(b + o_out);
  s->d_len = reinterpret_cast<int64_t*>(b + o_len);
  return TT_OK;
}

int ws_reserve_docs(Workspace* s, int64_t n_docs, hipStream_t st) {
  if (n_docs + 1 <= s->doc_cap) return TT_OK;
  if (s->d_docs && hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
  if (s->d_docs) (void)hipFree(s->d_docs);
  s->d_docs = nullptr;
  s->doc_cap = 0;
  int64_t cap = std::max<int64_t>(n_docs + 1, 64);
  void* m = nullptr;
  if (hipMalloc(&m, 2 * 8 * cap) != hipSuccess) return TT_ERR_OOM;
  s->d_docs = static_cast<int64_t*>(m);
  s->d_out_docs = s->d_docs + cap;
  s->doc_cap = cap;
  return TT_OK;
}

int get_ws(tt_tokenizer* h, hipStream_t stream, uint64_t need, Workspace** out) {
  Workspace* s;
  {
    std::lock_guard<std::mutex> g(h->mu);
    auto it = h->ws.find(stream);
    if (it == h->ws.end()) {
      s = new Workspace();
      if (hipHostMalloc(reinterpret_cast<void**>(&s->h_len), 8, hipHostMallocDefault) != hipSuccess) {
        free_ws(s);
        return TT_ERR_OOM;
      }
      h->ws[stream] = s;
    } else {
      s = it->second;
    }
  }
  int rc = ws_reserve(s, need, stream);
  if (rc) return rc;
  *out = s;
  return TT_OK;
}

// The spans buffer of a workspace (host span export), allocated on first use
// and grown with the workspace's capacity.
int reserve_spans(Workspace* s, uint64_t len, hipStream_t st) {
  if (len <= s->span_cap) return TT_OK;
  if (s->d_spans) {
    if (hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
    (void)hipFree(s->d_spans);
    s->d_spans = nullptr;
    s->span_cap = 0;
  }
  if (hipMalloc(reinterpret_cast<void**>(&s->d_spans), 16 * (size_t)s->cap) != hipSuccess) return TT_ERR_OOM;
  s->span_cap = s->cap;
  return TT_OK;
}

// The pinned staging buffers of tt_encode, allocated on first use and grown
// with the workspace's capacity (5 bytes per byte of capacity).  Only blocking
// calls use them, so none is in use when they grow.
int reserve_pinned(Workspace* s, uint64_t len) {
  if (len <= s->pin_cap) return TT_OK;
  auto drop = [&]() {
    if (s->h_in) (void)hipHostFree(s->h_in);
    if (s->h_ids) (void)hipHostFree(s->h_ids);
    s->h_in = nullptr;
    s->h_ids = nullptr;
    s->pin_cap = 0;
  };
  drop();
  const uint64_t cap = s->cap;  // >= len (the device workspace was reserved first)
  if (hipHostMalloc(reinterpret_cast<void**>(&s->h_in), cap + 64, hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc(reinterpret_cast<void**>(&s->h_ids), 4 * cap, hipHostMallocDefault) != hipSuccess) {
    drop();
    return TT_ERR_OOM;
  }
  s->pin_cap = cap;
  return TT_OK;
}

// Whether [p, p + len) is pinned host memory the device can read directly.
bool host_pinned(const void* p, int64_t len) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();  // pageable memory may report an error; it is not sticky
    return false;
  }
  if (a.type != hipMemoryTypeHost) return false;
  if (hipPointerGetAttributes(&a, static_cast<const uint8_t*>(p) + (len - 1)) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return a.type == hipMemoryTypeHost;
}

// Enqueue the whole chain for `n` bytes at device address `text`.
// mode 0: split export (out_ids receives piece offsets); mode 1: encode;
// mode 2: encode with span export into out_spans ([n][4], single requests).
int run_chain(tt_tokenizer* h, Workspace* s, const uint8_t* text, uint32_t n, const int64_t* d_docs,
              int32_t n_docs, int32_t* out_ids, int64_t* out_len, int64_t* out_docs, hipStream_t st, int mode,
              int32_t* out_spans = nullptr, uint16_t* out16 = nullptr, uint8_t* out_hi = nullptr) {
  if (s->epoch + 1 >= EPOCH_LIMIT) {
    // epochs wrapped: clear the words that carry them and start again
    if (hipMemsetAsync(s->dmem, 0, s->ctl_bytes, st) != hipSuccess) return TT_ERR_HIP;
    s->epoch = 0;
    s->ticket_base = 0;
  }
  Work w = s->w;
  w.text = text;
  w.n = n;
  w.doc_off = d_docs;
  w.n_docs = n_docs;
  w.epoch = ++s->epoch;
  w.ticket_base = s->ticket_base;
  w.n_tiles = n_tiles_for(n);
  w.out_ids = out_ids;
  w.out_len = out_len;
  w.out_doc_off = out_docs;
  w.out_spans = out_spans;
  w.out16 = mode == 1 ? out16 : nullptr;
  w.out_hi = mode == 1 && out16 ? out_hi : nullptr;
  const DevTables tb = handle_tables(h);
  const int ring = h->profile;
  if (ring != s->ring) {  // (re)size the event ring
    for (auto e : s->ev)
      if (e) (void)hipEventDestroy(e);
    s->ev.assign((size_t)ring * (N_STAGES + 1), nullptr);
    s->ring = ring;
    s->n_calls = 0;
  }
  hipEvent_t* evs = ring ? &s->ev[(size_t)(s->n_calls % ring) * (N_STAGES + 1)] : nullptr;
  int n_mark = 0;
  auto mark = [&]() -> bool {
    if (!ring) return true;
    hipEvent_t& e = evs[n_mark++];
    // timing only: no system-scope fence (no cache writeback) at each mark
    if (!e && hipEventCreateWithFlags(&e, hipEventDisableSystemFence) != hipSuccess) return false;
    return hipEventRecord(e, st) == hipSuccess;
  };
  if (!mark()) return TT_ERR_HIP;
  if (launch_tile(w, tb, h->pattern, mode, h->ignore && mode != 0, st) != hipSuccess) return TT_ERR_HIP;
  s->ticket_base += w.n_tiles;  // the tiles took their tickets
  if (d_docs && launch_doc_offsets(w, st) != hipSuccess) return TT_ERR_HIP;
  if (mode == 2 && launch_spans(w, st) != hipSuccess) return TT_ERR_HIP;
  if (!mark()) return TT_ERR_HIP;
  if (ring) ++s->n_calls;
  return TT_OK;
}

// Largest request that tt_encode stages through pinned buffers; longer ones
// are copied from and to the caller's memory directly.
constexpr uint64_t PINNED_MAX = 1ull << 28;

// tt_encode through pinned staging, with one host synchronisation.
//  - stage-in: the tile kernel reads the request straight from pinned host
//    memory (the caller's buffer when it is pinned, else a pinned copy): each
//    tile fetches its window over the bus as it starts, so the transfer
//    overlaps the tiles' work instead of preceding the launch;
//  - stage-out: the tile kernel places the IDs straight into pinned host
//    memory (the caller's array when it is pinned, else pinned staging that
//    the copy threads then copy into the caller's array), and its last tile
//    writes the output length there too: no copy engine transfer at all.
//    Each wave of a tile writes its IDs as one contiguous range (whole lines
//    over the bus).  Staged IDs of a handle whose caller IDs all fit in 16
//    bits cross the bus as 16-bit values (half the bytes), in 24 bits as a
//    16-bit array and an array of their third bytes (three quarters), and
//    the copy threads widen them into the caller's array.
int encode_staged(tt_tokenizer* h, Workspace* s, const uint8_t* utf8, int64_t len, int32_t* out_ids,
                  int64_t* out_len, hipStream_t st) {
  int rc = reserve_pinned(s, (uint64_t)len);
  if (rc) return rc;
  const uint8_t* src = utf8;
  const bool pin_out = host_pinned(out_ids, 4 * len);
  const bool pin_in = host_pinned(utf8, len);
  if (!pin_out || !pin_in) host_copy_wake((size_t)len);  // (the IDs take about as many bytes)
  if (!pin_in) {
    host_copy(s->h_in, utf8, (size_t)len);
    src = s->h_in;
  }
  *s->h_len = 0;
  // the tile kernel writes the IDs at their places in pinned host memory
  int32_t* dst = pin_out ? out_ids : s->h_ids;
  // narrow staging: the low 16 bits at the start of h_ids, the third bytes
  // after 2 * len bytes (3 * len <= the 4 * capacity bytes of h_ids)
  const bool narrow = !pin_out && h->id_bits < 32;
  uint16_t* lo16 = reinterpret_cast<uint16_t*>(s->h_ids);
  uint8_t* hi8 = narrow && h->id_bits == 24 ? reinterpret_cast<uint8_t*>(s->h_ids) + 2 * (size_t)len : nullptr;
  rc = run_chain(h, s, src, (uint32_t)len, nullptr, 0, dst, s->h_len, nullptr, st, 1, nullptr,
                 narrow ? lo16 : nullptr, hi8);
  if (rc) return rc;
  if (hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
  const int64_t T = *s->h_len;
  if (T < 0) return (int)T;
  if (T > len) return TT_ERR_HIP;  // cannot happen: at most one ID per byte
  if (!pin_out && T > 0) {
    if (narrow) host_widen(out_ids, lo16, hi8, (size_t)T);
    else host_copy(out_ids, s->h_ids, 4 * (size_t)T);
  }
  *out_len = T;
  return TT_OK;
}

// An entry of the whole-unit dictionaries: up to DICT2_MAX bytes as words.
struct DictEntry {
  uint32_t w[6], len, id;
};

DictEntry make_entry(const uint8_t* p, uint32_t L, uint32_t id) {
  DictEntry e{{0u, 0u, 0u, 0u, 0u, 0u}, L, id};
  for (uint32_t i = 0; i < L; ++i) e.w[i >> 2] |= (uint32_t)p[i] << (8 * (i & 3));
  return e;
}

// Two-choice cuckoo table of 2..DICT_MAX-byte strings, two entries per bucket,
// load 0.8; grows by 1/8 while an entry cannot be placed.  Returns nonzero if
// the table would not fit.
int build_dict(const std::vector<DictEntry>& entries, std::vector<u32x4>& dict, uint32_t& dnb) {
  dnb = (uint32_t)(entries.size() * 5 / 8) + 16;
  for (;;) {
    dict.assign(2 * (size_t)dnb, u32x4{0u, 0u, 0u, 0u});
    uint64_t rng = 0xD1B54A32D192ED03ull;
    bool ok = true;
    for (size_t i = 0; i < entries.size() && ok; ++i) {
      u32x4 item{entries[i].w[0], entries[i].w[1], entries[i].w[2], (entries[i].id << 4) | entries[i].len};
      ok = false;
      for (int kick = 0; kick < 2000; ++kick) {
        const uint32_t len = item.w & 15u;
        const size_t b1 = 2 * (size_t)bucket_of(unit_hash(item.x, item.y, item.z, len), dnb);
        const size_t b2 = 2 * (size_t)bucket_of(unit_hash2(item.x, item.y, item.z, len), dnb);
        size_t free_at = SIZE_MAX;
        for (size_t c : {b1, b1 + 1, b2, b2 + 1})
          if (dict[c].w == 0u) {
            free_at = c;
            break;
          }
        if (free_at != SIZE_MAX) {
          dict[free_at] = item;
          ok = true;
          break;
        }
        rng ^= rng << 13;
        rng ^= rng >> 7;
        rng ^= rng << 17;
        const size_t v = ((rng & 2) ? b1 : b2) + (rng & 1);
        std::swap(item, dict[v]);
      }
    }
    if (ok) return 0;
    dnb += dnb / 8;
    if (dnb > (1u << 27)) return 1;
  }
}

// Two-choice cuckoo table of DICT_MAX+1..DICT2_MAX-byte strings, one entry of
// two words per bucket, load below 1/2.
int build_dict2(const std::vector<DictEntry>& entries2, std::vector<u32x4>& dict2, uint32_t& dnb2) {
  dnb2 = (uint32_t)(entries2.size() * 2) + 16;
  for (;;) {
    dict2.assign(2 * (size_t)dnb2, u32x4{0u, 0u, 0u, 0u});
    uint64_t rng = 0x9E3779B97F4A7C15ull;
    bool ok = true;
    for (size_t i = 0; i < entries2.size() && ok; ++i) {
      const DictEntry* item = &entries2[i];
      DictEntry held;
      ok = false;
      for (int kick = 0; kick < 1000; ++kick) {
        const uint32_t* q = item->w;
        const size_t b1 = 2 * (size_t)bucket_of(unit_hash6(q[0], q[1], q[2], q[3], q[4], q[5], item->len), dnb2);
        const size_t b2 = 2 * (size_t)bucket_of(unit_hash6b(q[0], q[1], q[2], q[3], q[4], q[5], item->len), dnb2);
        const u32x4 x0{q[0], q[1], q[2], q[3]}, x1{q[4], q[5], (item->id << 5) | item->len, 0u};
        size_t at = SIZE_MAX;
        if (dict2[b1 + 1].z == 0u) at = b1;
        else if (dict2[b2 + 1].z == 0u) at = b2;
        if (at != SIZE_MAX) {
          dict2[at] = x0;
          dict2[at + 1] = x1;
          ok = true;
          break;
        }
        rng ^= rng << 13;
        rng ^= rng >> 7;
        rng ^= rng << 17;
        const size_t v = (rng & 1) ? b1 : b2;
        DictEntry out;
        out.w[0] = dict2[v].x;
        out.w[1] = dict2[v].y;
        out.w[2] = dict2[v].z;
        out.w[3] = dict2[v].w;
        out.w[4] = dict2[v + 1].x;
        out.w[5] = dict2[v + 1].y;
        out.len = dict2[v + 1].z & 31u;
        out.id = dict2[v + 1].z >> 5;
        dict2[v] = x0;
        dict2[v + 1] = x1;
        held = out;
        item = &held;
      }
    }
    if (ok) return 0;
    dnb2 += dnb2 / 8;
    if (dnb2 > (1u << 27)) return 1;
  }
}

}  // namespace

namespace {

// The batch chain over host documents, with the IDs and per-document output
// offsets copied back into host vectors (used by the added-token paths, whose
// documents are the text segments and the literals between them).
int batch_host(tt_tokenizer* h, hipStream_t st, const uint8_t* concat, int64_t len,
               const std::vector<int64_t>& docs, std::vector<int32_t>& ids, std::vector<int64_t>& out_docs) {
  const int64_t n_docs = (int64_t)docs.size() - 1;
  if (n_docs > INT32_MAX) return TT_ERR_TOO_LARGE;
  out_docs.assign(docs.size(), 0);
  ids.clear();
  if (len == 0) return TT_OK;
  if (hipSetDevice(h->device) != hipSuccess) return TT_ERR_HIP;
  Workspace* s = nullptr;
  int rc = get_ws(h, st, (uint64_t)len, &s);
  if (rc) return rc;
  rc = ws_reserve_docs(s, n_docs, st);
  if (rc) return rc;
  if (hipMemcpyAsync(s->d_in, concat, (size_t)len, hipMemcpyHostToDevice, st) != hipSuccess ||
      hipMemcpyAsync(s->d_docs, docs.data(), 8 * docs.size(), hipMemcpyHostToDevice, st) != hipSuccess)
    return TT_ERR_HIP;
  rc = run_chain(h, s, s->d_in, (uint32_t)len, s->d_docs, (int32_t)n_docs, s->d_out, s->d_len, s->d_out_docs, st, 1);
  if (rc) return rc;
  if (hipMemcpyAsync(s->h_len, s->d_len, 8, hipMemcpyDeviceToHost, st) != hipSuccess) return TT_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
  const int64_t T = *s->h_len;
  if (T < 0) return (int)T;
  if (T > len) return TT_ERR_HIP;  // cannot happen: at most one ID per byte
  ids.resize((size_t)std::max<int64_t>(T, 1));
  if (hipMemcpyAsync(ids.data(), s->d_out, (size_t)T * 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipMemcpyAsync(out_docs.data(), s->d_out_docs, 8 * docs.size(), hipMemcpyDeviceToHost, st) != hipSuccess)
    return TT_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
  ids.resize((size_t)T);
  return TT_OK;
}

// Documents of one text [a, b) of `t` around its added-token literals: text
// before the first literal, the literal, text up to the next literal, and so
// on (text documents may be empty); appends the boundaries after a to `docs`
// and the literals to `lits`.
void added_documents(const AddedSet& added, const uint8_t* t, int64_t a, int64_t b, std::vector<int64_t>& docs,
                     std::vector<AddedSet::Match>& lits) {
  std::vector<AddedSet::Match> m;
  added.extract(t + a, b - a, m);
  for (const auto& x : m) {
    docs.push_back(a + x.s);
    docs.push_back(a + x.e);
    lits.push_back(x);
  }
  docs.push_back(b);
}

}  // namespace

namespace tt {
int handle_pattern(const tt_tokenizer* h) { return h->pattern; }
int handle_device(const tt_tokenizer* h) { return h->device; }
bool handle_ignore(const tt_tokenizer* h) { return h->ignore; }
DevTables handle_tables(const tt_tokenizer* h) {
  return DevTables{h->d_slots, h->nb,     h->d_pair0,  h->d_join,  h->d_ext,   h->n_ids,
                   h->d_dict,  h->dnb,    h->d_dict2,  h->dnb2,    h->d_toklen, h->vmax,
                   h->d_vdict, h->vdnb,   h->d_vdict2, h->vdnb2,   h->d_vlong, h->vlnb,
                   h->d_vblob};
}
bool handle_has_added(const tt_tokenizer* h) { return !h->added.empty(); }
uint32_t handle_max_token_bytes(const tt_tokenizer* h) { return h->max_tok_bytes; }

// Span export of a small host request with one synchronisation: the length,
// and `len` ID and span slots (at least the T written, since T <= len), leave
// the device together.  h_in, h_ids, h_spans and h_len are pinned host memory
// of at least len, len, 4 len and 1 entries.
int encode_spans_pinned(tt_tokenizer* h, const uint8_t* h_in, int64_t len, int32_t* h_ids, int32_t* h_spans,
                        int64_t* h_len, void* stream) {
  if (!h || !h_in || !h_ids || !h_spans || !h_len) return TT_ERR_NULL_ARG;
  if (!h->added.empty()) return TT_ERR_BAD_ARG;
  if (len <= 0) return TT_ERR_BAD_ARG;
  if (len > TT_MAX_BYTES) return TT_ERR_TOO_LARGE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (hipSetDevice(h->device) != hipSuccess) return TT_ERR_HIP;
  Workspace* s = nullptr;
  int rc = get_ws(h, st, (uint64_t)len, &s);
  if (rc) return rc;
  rc = reserve_spans(s, (uint64_t)len, st);
  if (rc) return rc;
  if (hipMemcpyAsync(s->d_in, h_in, (size_t)len, hipMemcpyHostToDevice, st) != hipSuccess) return TT_ERR_HIP;
  rc = run_chain(h, s, s->d_in, (uint32_t)len, nullptr, 0, s->d_out, s->d_len, nullptr, st, 2, s->d_spans);
  if (rc) return rc;
  if (hipMemcpyAsync(h_len, s->d_len, 8, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipMemcpyAsync(h_ids, s->d_out, (size_t)len * 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipMemcpyAsync(h_spans, s->d_spans, (size_t)len * 16, hipMemcpyDeviceToHost, st) != hipSuccess)
    return TT_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
  const int64_t T = *h_len;
  if (T < 0) return (int)T;
  if (T > len) return TT_ERR_HIP;  // cannot happen: at most one ID per byte
  return TT_OK;
}
}  // namespace tt

extern "C" {

const char* tt_status_string(int status) {
  switch (status) {
    case TT_OK: return "ok";
    case TT_ERR_NULL_ARG: return "a required pointer is NULL";
    case TT_ERR_BAD_PATTERN: return "unknown pattern id";
    case TT_ERR_BAD_MERGES: return "merge table out of range, duplicated or not proper";
    case TT_ERR_BAD_VOCAB: return "vocabulary inconsistent with the merges";
    case TT_ERR_INVALID_UTF8: return "input is not valid UTF-8";
    case TT_ERR_TOO_LARGE: return "request larger than TT_MAX_BYTES";
    case TT_ERR_HIP: return "HIP runtime error";
    case TT_ERR_OOM: return "out of memory";
    case TT_ERR_BAD_ARG: return "inconsistent size or offset argument";
    default: return "unknown status";
  }
}

int tt_create(const tt_merge* merges, int32_t n_merges, const uint8_t* vocab_bytes,
              const int64_t* vocab_offsets, int32_t vocab_size, int32_t pattern_id, tt_tokenizer** out) {
  return tt_create_ex(merges, n_merges, vocab_bytes, vocab_offsets, vocab_size, pattern_id, nullptr, out);
}

int tt_create_ex(const tt_merge* merges, int32_t n_merges, const uint8_t* vocab_bytes,
                 const int64_t* vocab_offsets, int32_t vocab_size, int32_t pattern_id, const tt_options* opt,
                 tt_tokenizer** out) {
  if (!out || !vocab_offsets || (n_merges > 0 && !merges)) return TT_ERR_NULL_ARG;
  *out = nullptr;
  if (pattern_id != TT_PATTERN_GPT2 && pattern_id != TT_PATTERN_CL100K && pattern_id != TT_PATTERN_O200K &&
      pattern_id != TT_PATTERN_DEEPSEEK) return TT_ERR_BAD_PATTERN;
  const bool ignore = opt && opt->ignore_merges != 0;
  // added tokens: non-empty, strict UTF-8, bounded, distinct, non-negative IDs
  AddedSet added;
  if (opt && opt->n_added != 0) {
    if (opt->n_added < 0) return TT_ERR_BAD_ARG;
    if (!opt->added_bytes || !opt->added_offsets || !opt->added_ids) return TT_ERR_NULL_ARG;
    if (opt->added_offsets[0] != 0) return TT_ERR_BAD_ARG;
    std::unordered_set<std::string> lits;
    for (int32_t i = 0; i < opt->n_added; ++i) {
      const int64_t a = opt->added_offsets[i], b = opt->added_offsets[i + 1];
      if (b <= a || b - a > TT_MAX_ADDED_BYTES || opt->added_ids[i] < 0) return TT_ERR_BAD_ARG;
      std::string lit(reinterpret_cast<const char*>(opt->added_bytes + a), (size_t)(b - a));
      if (!valid_utf8(reinterpret_cast<const uint8_t*>(lit.data()), (int64_t)lit.size())) return TT_ERR_BAD_ARG;
      if (!lits.insert(lit).second) return TT_ERR_BAD_ARG;
      added.add(lit, opt->added_ids[i]);
    }
    added.finish();
  }
  if (n_merges < 0 || vocab_size < 256 || (uint32_t)n_merges > MAX_MERGES) return TT_ERR_BAD_ARG;
  if (vocab_offsets[0] != 0) return TT_ERR_BAD_VOCAB;
  for (int32_t i = 0; i < vocab_size; ++i)
    if (vocab_offsets[i + 1] < vocab_offsets[i]) return TT_ERR_BAD_VOCAB;
  if (vocab_offsets[vocab_size] > 0 && !vocab_bytes) return TT_ERR_NULL_ARG;
  auto vlen = [&](int32_t id) { return vocab_offsets[id + 1] - vocab_offsets[id]; };
  auto vptr = [&](int32_t id) { return vocab_bytes + vocab_offsets[id]; };

  // base IDs: lowest ID spelling each single byte
  std::vector<int32_t> byte_id(256, -1);
  for (int32_t i = 0; i < vocab_size; ++i)
    if (vlen(i) == 1 && byte_id[vptr(i)[0]] < 0) byte_id[vptr(i)[0]] = i;
  for (int b = 0; b < 256; ++b)
    if (byte_id[b] < 0) return TT_ERR_BAD_VOCAB;

  // properness: operands available before use, results fresh and unique.
  // internal[] gives the library's ID of every available vocabulary ID: byte b
  // is b, the result of merge r is 256 + r
  std::vector<int32_t> internal(vocab_size, -1);
  for (int b = 0; b < 256; ++b) internal[byte_id[b]] = b;
  std::unordered_set<uint64_t> pairs;
  pairs.reserve((size_t)n_merges * 2 + 16);
  for (int32_t r = 0; r < n_merges; ++r) {
    const tt_merge& m = merges[r];
    if (m.left < 0 || m.right < 0 || m.result < 0 || m.left >= vocab_size || m.right >= vocab_size ||
        m.result >= vocab_size)
      return TT_ERR_BAD_MERGES;
    uint64_t key = ((uint64_t)(uint32_t)m.left << 32) | (uint32_t)m.right;
    if (!pairs.insert(key).second) return TT_ERR_BAD_MERGES;
    if (internal[m.left] < 0 || internal[m.right] < 0 || internal[m.result] >= 0) return TT_ERR_BAD_MERGES;
    int64_t la = vlen(m.left), lb = vlen(m.right);
    if (vlen(m.result) != la + lb || std::memcmp(vptr(m.result), vptr(m.left), la) != 0 ||
        std::memcmp(vptr(m.result) + la, vptr(m.right), lb) != 0)
      return TT_ERR_BAD_VOCAB;
    internal[m.result] = 256 + r;
  }
  // under ignore_merges every other vocabulary ID becomes reachable (a piece
  // can be that entry): internal IDs 256 + M + j follow the merge results
  std::vector<int32_t> extras;
  if (ignore)
    for (int32_t i = 0; i < vocab_size; ++i)
      if (internal[i] < 0) {
        internal[i] = (int32_t)(256 + n_merges + (int32_t)extras.size());
        extras.push_back(i);
      }
  const uint32_t n_ids = 256u + (uint32_t)n_merges + (uint32_t)extras.size();
  std::vector<int32_t> ext(n_ids);
  for (int b = 0; b < 256; ++b) ext[b] = byte_id[b];
  for (int32_t r = 0; r < n_merges; ++r) ext[256 + r] = merges[r].result;
  for (size_t j = 0; j < extras.size(); ++j) ext[256 + (size_t)n_merges + j] = extras[j];
  // byte length of every internal ID (span export): a merge result spells its
  // operands back to back, and both operands come before it
  std::vector<uint32_t> toklen(n_ids, 1u);
  for (int32_t r = 0; r < n_merges; ++r) {
    const uint64_t l = (uint64_t)toklen[(size_t)internal[merges[r].left]] + toklen[(size_t)internal[merges[r].right]];
    toklen[256 + (size_t)r] = l > 0xFFFFFFFFull ? 0xFFFFFFFFu : (uint32_t)l;
  }
  for (size_t j = 0; j < extras.size(); ++j) {
    const int64_t l = vlen(extras[j]);
    toklen[256 + (size_t)n_merges + j] = l > 0xFFFFFFFFll ? 0xFFFFFFFFu : (uint32_t)l;
  }

  // byte-pair ranks, and the two-choice cuckoo table of all pairs (two slots
  // per bucket, load 0.8; the table grows by 1/8 while an insertion cannot be
  // placed)
  std::vector<uint32_t> pair0(65536, RANK_INF);
  for (int32_t r = 0; r < n_merges; ++r) {
    const int32_t a = internal[merges[r].left], b = internal[merges[r].right];
    if (a < 256 && b < 256) pair0[((uint32_t)a << 8) | (uint32_t)b] = (uint32_t)r;
  }
  uint32_t nb = (uint32_t)((uint64_t)n_merges * 5 / 8) + 16;
  std::vector<uint64_t> slots;
  for (;;) {
    slots.assign(2 * (size_t)nb, SLOT_EMPTY);
    uint64_t rng = 0x9E3779B97F4A7C15ull;
    bool ok = true;
    for (int32_t r = 0; r < n_merges && ok; ++r) {
      uint64_t item = slot_key((uint32_t)internal[merges[r].left], (uint32_t)internal[merges[r].right]) |
                      ((uint64_t)r << (2 * ID_BITS));
      ok = false;
      for (int kick = 0; kick < 1000; ++kick) {
        const uint32_t a = (uint32_t)(item & ID_LIMIT), b = (uint32_t)((item >> ID_BITS) & ID_LIMIT);
        const uint32_t b1 = bucket_of(pair_hash(a, b), nb), b2 = bucket_of(pair_hash2(a, b), nb);
        size_t free_at = SIZE_MAX;
        for (size_t c : {2 * (size_t)b1, 2 * (size_t)b1 + 1, 2 * (size_t)b2, 2 * (size_t)b2 + 1})
          if (slots[c] == SLOT_EMPTY) {
            free_at = c;
            break;
          }
        if (free_at != SIZE_MAX) {
          slots[free_at] = item;
          ok = true;
          break;
        }
        rng ^= rng << 13;
        rng ^= rng >> 7;
        rng ^= rng << 17;
        const size_t victim = 2 * (size_t)((rng & 2) ? b1 : b2) + (rng & 1);
        std::swap(item, slots[victim]);
      }
    }
    if (ok) break;
    nb += nb / 8;
    if (nb > (1u << 28)) return TT_ERR_OOM;
  }

  // whole-unit dictionaries: every byte string of 3..DICT2_MAX bytes that is
  // the spelling of a merge result and whose BPE (computed here, exactly as the
  // device computes it) is that single token; strings of up to DICT_MAX bytes
  // go to the first, longer ones to the second
  std::vector<u32x4> dict, dict2;
  uint32_t dnb = 16, dnb2 = 16;
  {
    std::unordered_map<uint64_t, uint32_t> rank;
    rank.reserve((size_t)n_merges * 2 + 16);
    for (int32_t r = 0; r < n_merges; ++r)
      rank.emplace(slot_key((uint32_t)internal[merges[r].left], (uint32_t)internal[merges[r].right]), (uint32_t)r);
    auto lookup = [&](uint32_t a, uint32_t b) -> uint32_t {
      auto it = rank.find(slot_key(a, b));
      return it == rank.end() ? RANK_INF : it->second;
    };
    std::vector<DictEntry> entries, entries2;
    std::unordered_set<std::string> seen;
    uint32_t ids[DICT2_MAX], rk[DICT2_MAX];
    for (int32_t r = 0; r < n_merges; ++r) {
      const int32_t res = merges[r].result;
      const int64_t L = vlen(res);
      if (L < 3 || L > DICT2_MAX) continue;
      std::string key(reinterpret_cast<const char*>(vptr(res)), (size_t)L);
      if (!seen.insert(key).second) continue;
      // greedy lowest-rank BPE of the spelling, leftmost among equal ranks
      int n = (int)L;
      for (int i = 0; i < n; ++i) ids[i] = vptr(res)[i];
      for (int i = 0; i + 1 < n; ++i) rk[i] = lookup(ids[i], ids[i + 1]);
      while (n > 1) {
        int k = -1;
        uint32_t best = RANK_INF;
        for (int i = 0; i + 1 < n; ++i)
          if (rk[i] < best) {
            best = rk[i];
            k = i;
          }
        if (k < 0) break;
        ids[k] = 256u + best;
        for (int i = k + 1; i + 1 < n; ++i) {
          ids[i] = ids[i + 1];
          rk[i] = rk[i + 1];
        }
        --n;
        rk[k] = k + 1 < n ? lookup(ids[k], ids[k + 1]) : RANK_INF;
        if (k > 0) rk[k - 1] = lookup(ids[k - 1], ids[k]);
      }
      if (n != 1) continue;
      (L <= DICT_MAX ? entries : entries2).push_back(make_entry(vptr(res), (uint32_t)L, ids[0]));
    }
    if (build_dict(entries, dict, dnb) || build_dict2(entries2, dict2, dnb2)) return TT_ERR_OOM;
  }

  // ignore_merges: every vocabulary string of at least two bytes, with the
  // internal ID of its lowest vocabulary ID, in tables by length
  std::vector<u32x4> vdict, vdict2, vlong;
  std::vector<uint8_t> vblob;
  uint32_t vdnb = 0, vdnb2 = 0, vlnb = 0, vmax = 0;
  if (ignore) {
    std::vector<DictEntry> e1, e2;
    std::vector<std::pair<int32_t, uint32_t>> longs;  // (vocabulary ID, internal ID)
    std::unordered_set<std::string> seen;
    for (int32_t i = 0; i < vocab_size; ++i) {
      const int64_t L = vlen(i);
      if (L < 2) continue;
      if (!seen.insert(std::string(reinterpret_cast<const char*>(vptr(i)), (size_t)L)).second) continue;
      vmax = std::max<uint32_t>(vmax, (uint32_t)std::min<int64_t>(L, 0x7FFFFFFF));
      if (L <= DICT_MAX) e1.push_back(make_entry(vptr(i), (uint32_t)L, (uint32_t)internal[i]));
      else if (L <= DICT2_MAX) e2.push_back(make_entry(vptr(i), (uint32_t)L, (uint32_t)internal[i]));
      else longs.emplace_back(i, (uint32_t)internal[i]);
    }
    vmax = std::max<uint32_t>(vmax, 2u);
    if (build_dict(e1, vdict, vdnb) || build_dict2(e2, vdict2, vdnb2)) return TT_ERR_OOM;
    // longer strings: cuckoo buckets of two {hash, length, ID, offset} slots
    vlnb = (uint32_t)(longs.size() * 5 / 8) + 16;
    for (;;) {
      vlong.assign(2 * (size_t)vlnb, u32x4{0u, 0u, 0u, 0u});
      vblob.clear();
      uint64_t rng = 0x2545F4914F6CDD1Dull;
      bool ok = true;
      for (size_t k = 0; k < longs.size() && ok; ++k) {
        const int32_t vid = longs[k].first;
        const uint32_t L = (uint32_t)vlen(vid);
        uint32_t h1 = LONG_SEED1, h2 = LONG_SEED2;
        for (uint32_t j = 0; j < L; ++j) {
          h1 = long_hash_step(h1, vptr(vid)[j]);
          h2 = long_hash_step(h2, vptr(vid)[j]);
        }
        h1 = long_hash_final(h1, L);
        h2 = long_hash_final(h2, L);
        const uint32_t off = (uint32_t)vblob.size();
        vblob.insert(vblob.end(), vptr(vid), vptr(vid) + L);
        // (the bucket choice of a displaced entry is recomputed from its bytes)
        u32x4 item{h1, L, longs[k].second, off};
        ok = false;
        for (int kick = 0; kick < 1000; ++kick) {
          uint32_t g1 = LONG_SEED1, g2 = LONG_SEED2;
          for (uint32_t j = 0; j < item.y; ++j) {
            g1 = long_hash_step(g1, vblob[item.w + j]);
            g2 = long_hash_step(g2, vblob[item.w + j]);
          }
          const size_t b1 = 2 * (size_t)bucket_of(long_hash_final(g1, item.y), vlnb);
          const size_t b2 = 2 * (size_t)bucket_of(long_hash_final(g2, item.y), vlnb);
          size_t free_at = SIZE_MAX;
          for (size_t c : {b1, b1 + 1, b2, b2 + 1})
            if (vlong[c].y == 0u) {
              free_at = c;
              break;
            }
          if (free_at != SIZE_MAX) {
            vlong[free_at] = item;
            ok = true;
            break;
          }
          rng ^= rng << 13;
          rng ^= rng >> 7;
          rng ^= rng << 17;
          const size_t v = ((rng & 2) ? b1 : b2) + (rng & 1);
          std::swap(item, vlong[v]);
        }
      }
      if (ok) break;
      vlnb += vlnb / 8;
      if (vlnb > (1u << 27)) return TT_ERR_OOM;
    }
    if (vblob.empty()) vblob.push_back(0);
  }

  // junction byte pairs: the first merge that ever joins across a byte
  // boundary has its junction exactly there, so a boundary whose byte pair is
  // no merge's junction is never crossed
  std::vector<uint32_t> join(2048, 0u);
  for (int32_t r = 0; r < n_merges; ++r) {
    if (vlen(merges[r].left) == 0 || vlen(merges[r].right) == 0) continue;
    uint32_t x = vptr(merges[r].left)[vlen(merges[r].left) - 1];
    uint32_t y = vptr(merges[r].right)[0];
    uint32_t key = (x << 8) | y;
    join[key >> 5] |= 1u << (key & 31u);
  }

  tt_tokenizer* h = new tt_tokenizer();
  h->pattern = pattern_id;
  h->ignore = ignore;
  h->vmax = vmax;
  h->vdnb = vdnb;
  h->vdnb2 = vdnb2;
  h->vlnb = vlnb;
  h->added = std::move(added);
  h->n_merges = n_merges;
  h->vocab_size = vocab_size;
  h->nb = nb;
  h->dnb = dnb;
  h->dnb2 = dnb2;
  h->n_ids = n_ids;
  const int32_t ext_max = *std::max_element(ext.begin(), ext.end());
  const bool ext_nonneg = *std::min_element(ext.begin(), ext.end()) >= 0;
  h->id_bits = !ext_nonneg ? 32 : ext_max < (1 << 16) ? 16 : ext_max < (1 << 24) ? 24 : 32;
  h->max_tok_bytes = *std::max_element(toklen.begin(), toklen.end());
  if (hipGetDevice(&h->device) != hipSuccess) {
    delete h;
    return TT_ERR_HIP;
  }
  if (hipMalloc(reinterpret_cast<void**>(&h->d_slots), 16 * (size_t)nb) != hipSuccess ||
      hipMalloc(reinterpret_cast<void**>(&h->d_pair0), sizeof(uint32_t) * 65536) != hipSuccess ||
      hipMalloc(reinterpret_cast<void**>(&h->d_dict), sizeof(u32x4) * dict.size()) != hipSuccess ||
      hipMalloc(reinterpret_cast<void**>(&h->d_dict2), sizeof(u32x4) * dict2.size()) != hipSuccess ||
      hipMalloc(reinterpret_cast<void**>(&h->d_ext), sizeof(int32_t) * n_ids) != hipSuccess ||
      hipMalloc(reinterpret_cast<void**>(&h->d_toklen), sizeof(uint32_t) * n_ids) != hipSuccess ||
      hipMalloc(reinterpret_cast<void**>(&h->d_join), sizeof(uint32_t) * 2048) != hipSuccess) {
    tt_destroy(h);
    return TT_ERR_OOM;
  }
  if (ignore && (hipMalloc(reinterpret_cast<void**>(&h->d_vdict), sizeof(u32x4) * vdict.size()) != hipSuccess ||
                 hipMalloc(reinterpret_cast<void**>(&h->d_vdict2), sizeof(u32x4) * vdict2.size()) != hipSuccess ||
                 hipMalloc(reinterpret_cast<void**>(&h->d_vlong), sizeof(u32x4) * vlong.size()) != hipSuccess ||
                 hipMalloc(reinterpret_cast<void**>(&h->d_vblob), vblob.size()) != hipSuccess)) {
    tt_destroy(h);
    return TT_ERR_OOM;
  }
  if (ignore &&
      (hipMemcpy(h->d_vdict, vdict.data(), sizeof(u32x4) * vdict.size(), hipMemcpyHostToDevice) != hipSuccess ||
       hipMemcpy(h->d_vdict2, vdict2.data(), sizeof(u32x4) * vdict2.size(), hipMemcpyHostToDevice) != hipSuccess ||
       hipMemcpy(h->d_vlong, vlong.data(), sizeof(u32x4) * vlong.size(), hipMemcpyHostToDevice) != hipSuccess ||
       hipMemcpy(h->d_vblob, vblob.data(), vblob.size(), hipMemcpyHostToDevice) != hipSuccess)) {
    tt_destroy(h);
    return TT_ERR_HIP;
  }
  if (hipMemcpy(h->d_slots, slots.data(), 16 * (size_t)nb, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(h->d_pair0, pair0.data(), sizeof(uint32_t) * 65536, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(h->d_dict, dict.data(), sizeof(u32x4) * dict.size(), hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(h->d_dict2, dict2.data(), sizeof(u32x4) * dict2.size(), hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(h->d_ext, ext.data(), sizeof(int32_t) * n_ids, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(h->d_toklen, toklen.data(), sizeof(uint32_t) * n_ids, hipMemcpyHostToDevice) != hipSuccess ||
      hipMemcpy(h->d_join, join.data(), sizeof(uint32_t) * 2048, hipMemcpyHostToDevice) != hipSuccess) {
    tt_destroy(h);
    return TT_ERR_HIP;
  }
  *out = h;
  return TT_OK;
}

void tt_destroy(tt_tokenizer* h) {
  if (!h) return;
  (void)hipSetDevice(h->device);
  (void)hipDeviceSynchronize();
  for (auto& kv : h->ws) free_ws(kv.second);
  if (h->d_slots) (void)hipFree(h->d_slots);
  if (h->d_ext) (void)hipFree(h->d_ext);
  if (h->d_pair0) (void)hipFree(h->d_pair0);
  if (h->d_dict) (void)hipFree(h->d_dict);
  if (h->d_dict2) (void)hipFree(h->d_dict2);
  if (h->d_toklen) (void)hipFree(h->d_toklen);
  if (h->d_join) (void)hipFree(h->d_join);
  if (h->d_vdict) (void)hipFree(h->d_vdict);
  if (h->d_vdict2) (void)hipFree(h->d_vdict2);
  if (h->d_vlong) (void)hipFree(h->d_vlong);
  if (h->d_vblob) (void)hipFree(h->d_vblob);
  delete h;
}

int tt_info(const tt_tokenizer* h, int32_t* n_merges, int32_t* vocab_size, int32_t* pattern_id) {
  if (!h) return TT_ERR_NULL_ARG;
  if (n_merges) *n_merges = h->n_merges;
  if (vocab_size) *vocab_size = h->vocab_size;
  if (pattern_id) *pattern_id = h->pattern;
  return TT_OK;
}

int tt_encode_device(tt_tokenizer* h, const uint8_t* d_utf8, int64_t len, int32_t* d_out_ids,
                     int64_t* d_out_len, void* stream) {
  if (!h || !d_out_len || (len > 0 && (!d_utf8 || !d_out_ids))) return TT_ERR_NULL_ARG;
  if (!h->added.empty()) return TT_ERR_BAD_ARG;  // literals are extracted by the host entry points
  if (len < 0) return TT_ERR_BAD_ARG;
  if (len > TT_MAX_BYTES) return TT_ERR_TOO_LARGE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (hipSetDevice(h->device) != hipSuccess) return TT_ERR_HIP;
  if (len == 0) {
    static const int64_t zero = 0;
    return hipMemcpyAsync(d_out_len, &zero, 8, hipMemcpyHostToDevice, st) == hipSuccess ? TT_OK : TT_ERR_HIP;
  }
  Workspace* s = nullptr;
  int rc = get_ws(h, st, (uint64_t)len, &s);
  if (rc) return rc;
  return run_chain(h, s, d_utf8, (uint32_t)len, nullptr, 0, d_out_ids, d_out_len, nullptr, st, 1);
}

int tt_encode(tt_tokenizer* h, const uint8_t* utf8, int64_t len, int32_t* out_ids, int64_t* out_len,
              void* stream) {
  if (!h || !out_len || (len > 0 && (!utf8 || !out_ids))) return TT_ERR_NULL_ARG;
  if (len < 0) return TT_ERR_BAD_ARG;
  if (len > TT_MAX_BYTES) return TT_ERR_TOO_LARGE;
  *out_len = 0;
  if (len == 0) return TT_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (!h->added.empty()) {
    // literals first (host, leftmost-longest); the text segments and the
    // literals are the documents of one batch, and a literal's document is
    // replaced by its ID
    std::vector<int64_t> docs{0};
    std::vector<AddedSet::Match> lits;
    added_documents(h->added, utf8, 0, len, docs, lits);
    if (!lits.empty()) {
      std::vector<int32_t> ids;
      std::vector<int64_t> od;
      int rc = batch_host(h, st, utf8, len, docs, ids, od);
      if (rc) return rc;
      int64_t T = 0;
      for (size_t j = 0; j + 1 < docs.size(); ++j) {
        if (j & 1) {
          out_ids[T++] = lits[j / 2].id;
        } else {
          const int64_t c = od[j + 1] - od[j];
          if (c > 0) std::memcpy(out_ids + T, ids.data() + od[j], 4 * (size_t)c);
          T += c;
        }
      }
      *out_len = T;
      return TT_OK;
    }
  }
  if (hipSetDevice(h->device) != hipSuccess) return TT_ERR_HIP;
  Workspace* s = nullptr;
  int rc = get_ws(h, st, (uint64_t)len, &s);
  if (rc) return rc;
  if ((uint64_t)len <= PINNED_MAX) return encode_staged(h, s, utf8, len, out_ids, out_len, st);
  // very long requests: the length, then the IDs, straight between the caller's
  // memory and the device
  if (hipMemcpyAsync(s->d_in, utf8, (size_t)len, hipMemcpyHostToDevice, st) != hipSuccess) return TT_ERR_HIP;
  rc = run_chain(h, s, s->d_in, (uint32_t)len, nullptr, 0, s->d_out, s->d_len, nullptr, st, 1);
  if (rc) return rc;
  if (hipMemcpyAsync(s->h_len, s->d_len, 8, hipMemcpyDeviceToHost, st) != hipSuccess) return TT_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
  int64_t T = *s->h_len;
  if (T < 0) return (int)T;
  if (T > len) return TT_ERR_HIP;  // cannot happen: at most one ID per byte
  if (T > 0) {
    if (hipMemcpyAsync(out_ids, s->d_out, (size_t)T * 4, hipMemcpyDeviceToHost, st) != hipSuccess)
      return TT_ERR_HIP;
    if (hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
  }
  *out_len = T;
  return TT_OK;
}

int tt_encode_spans_device(tt_tokenizer* h, const uint8_t* d_utf8, int64_t len, int32_t* d_out_ids,
                           int32_t* d_out_spans, int64_t* d_out_len, void* stream) {
  if (!h || !d_out_len || (len > 0 && (!d_utf8 || !d_out_ids || !d_out_spans))) return TT_ERR_NULL_ARG;
  if (!h->added.empty()) return TT_ERR_BAD_ARG;  // literals are extracted by the host entry points
  if (len < 0) return TT_ERR_BAD_ARG;
  if (len > TT_MAX_BYTES) return TT_ERR_TOO_LARGE;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (hipSetDevice(h->device) != hipSuccess) return TT_ERR_HIP;
  if (len == 0) {
    static const int64_t zero = 0;
    return hipMemcpyAsync(d_out_len, &zero, 8, hipMemcpyHostToDevice, st) == hipSuccess ? TT_OK : TT_ERR_HIP;
  }
  Workspace* s = nullptr;
  int rc = get_ws(h, st, (uint64_t)len, &s);
  if (rc) return rc;
  return run_chain(h, s, d_utf8, (uint32_t)len, nullptr, 0, d_out_ids, d_out_len, nullptr, st, 2, d_out_spans);
}

int tt_encode_spans(tt_tokenizer* h, const uint8_t* utf8, int64_t len, int32_t* out_ids, int32_t* out_spans,
                    int64_t* out_len, void* stream) {
  if (!h || !out_len || (len > 0 && (!utf8 || !out_ids || !out_spans))) return TT_ERR_NULL_ARG;
  if (!h->added.empty()) return TT_ERR_BAD_ARG;  // literals are extracted by the host entry points
  if (len < 0) return TT_ERR_BAD_ARG;
  if (len > TT_MAX_BYTES) return TT_ERR_TOO_LARGE;
  *out_len = 0;
  if (len == 0) return TT_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (hipSetDevice(h->device) != hipSuccess) return TT_ERR_HIP;
  Workspace* s = nullptr;
  int rc = get_ws(h, st, (uint64_t)len, &s);
  if (rc) return rc;
  rc = reserve_spans(s, (uint64_t)len, st);
  if (rc) return rc;
  if (hipMemcpyAsync(s->d_in, utf8, (size_t)len, hipMemcpyHostToDevice, st) != hipSuccess) return TT_ERR_HIP;
  rc = run_chain(h, s, s->d_in, (uint32_t)len, nullptr, 0, s->d_out, s->d_len, nullptr, st, 2, s->d_spans);
  if (rc) return rc;
  if (hipMemcpyAsync(s->h_len, s->d_len, 8, hipMemcpyDeviceToHost, st) != hipSuccess) return TT_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
  const int64_t T = *s->h_len;
  if (T < 0) return (int)T;
  if (T > len) return TT_ERR_HIP;  // cannot happen: at most one ID per byte
  if (T > 0) {
    // IDs and spans leave the device back to back, with one synchronisation
    if (hipMemcpyAsync(out_ids, s->d_out, (size_t)T * 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
        hipMemcpyAsync(out_spans, s->d_spans, (size_t)T * 16, hipMemcpyDeviceToHost, st) != hipSuccess)
      return TT_ERR_HIP;
    if (hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
  }
  *out_len = T;
  return TT_OK;
}

int tt_encode_batch(tt_tokenizer* h, const uint8_t* concat, const int64_t* doc_offsets, int32_t n_docs,
                    int32_t* out_ids, int64_t* out_doc_offsets, void* stream) {
  if (!h || !doc_offsets || !out_doc_offsets) return TT_ERR_NULL_ARG;
  if (n_docs < 0 || doc_offsets[0] != 0) return TT_ERR_BAD_ARG;
  for (int32_t j = 0; j < n_docs; ++j)
    if (doc_offsets[j + 1] < doc_offsets[j]) return TT_ERR_BAD_ARG;
  const int64_t len = doc_offsets[n_docs];
  if (len > TT_MAX_BYTES) return TT_ERR_TOO_LARGE;
  if (len > 0 && (!concat || !out_ids)) return TT_ERR_NULL_ARG;
  if (len == 0) {
    for (int32_t j = 0; j <= n_docs; ++j) out_doc_offsets[j] = 0;
    return TT_OK;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (!h->added.empty()) {
    // every caller document becomes its text segments and literals
    std::vector<int64_t> docs{0};
    std::vector<AddedSet::Match> lits;
    std::vector<int64_t> first_doc((size_t)n_docs + 1), first_lit((size_t)n_docs + 1);
    for (int32_t d = 0; d < n_docs; ++d) {
      first_doc[(size_t)d] = (int64_t)docs.size() - 1;
      first_lit[(size_t)d] = (int64_t)lits.size();
      added_documents(h->added, concat, doc_offsets[d], doc_offsets[d + 1], docs, lits);
    }
    first_doc[(size_t)n_docs] = (int64_t)docs.size() - 1;
    first_lit[(size_t)n_docs] = (int64_t)lits.size();
    std::vector<int32_t> ids;
    std::vector<int64_t> od;
    int rc = batch_host(h, st, concat, len, docs, ids, od);
    if (rc) return rc;
    int64_t T = 0;
    for (int32_t d = 0; d < n_docs; ++d) {
      out_doc_offsets[d] = T;
      for (int64_t j = first_doc[(size_t)d]; j < first_doc[(size_t)d + 1]; ++j) {
        if ((j - first_doc[(size_t)d]) & 1) {
          out_ids[T++] = lits[(size_t)(first_lit[(size_t)d] + (j - first_doc[(size_t)d]) / 2)].id;
        } else {
          const int64_t c = od[(size_t)j + 1] - od[(size_t)j];
          if (c > 0) std::memcpy(out_ids + T, ids.data() + od[(size_t)j], 4 * (size_t)c);
          T += c;
        }
      }
    }
    out_doc_offsets[n_docs] = T;
    return TT_OK;
  }
  if (hipSetDevice(h->device) != hipSuccess) return TT_ERR_HIP;
  Workspace* s = nullptr;
  int rc = get_ws(h, st, (uint64_t)len, &s);
  if (rc) return rc;
  rc = ws_reserve_docs(s, n_docs, st);
  if (rc) return rc;
  if (hipMemcpyAsync(s->d_in, concat, (size_t)len, hipMemcpyHostToDevice, st) != hipSuccess) return TT_ERR_HIP;
  if (hipMemcpyAsync(s->d_docs, doc_offsets, 8 * ((size_t)n_docs + 1), hipMemcpyHostToDevice, st) != hipSuccess)
    return TT_ERR_HIP;
  rc = run_chain(h, s, s->d_in, (uint32_t)len, s->d_docs, n_docs, s->d_out, s->d_len, s->d_out_docs, st, 1);
  if (rc) return rc;
  if (hipMemcpyAsync(s->h_len, s->d_len, 8, hipMemcpyDeviceToHost, st) != hipSuccess) return TT_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
  int64_t T = *s->h_len;
  if (T < 0) return (int)T;
  if (T > len) return TT_ERR_HIP;  // cannot happen: at most one ID per byte
  if (hipMemcpyAsync(out_ids, s->d_out, (size_t)T * 4, hipMemcpyDeviceToHost, st) != hipSuccess ||
      hipMemcpyAsync(out_doc_offsets, s->d_out_docs, 8 * ((size_t)n_docs + 1), hipMemcpyDeviceToHost, st) !=
          hipSuccess)
    return TT_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
  return TT_OK;
}

int tt_pretokenize(tt_tokenizer* h, const uint8_t* utf8, int64_t len, int64_t* out_piece_starts, int64_t* out_n,
                   void* stream) {
  if (!h || !out_n || (len > 0 && (!utf8 || !out_piece_starts))) return TT_ERR_NULL_ARG;
  if (!h->added.empty()) return TT_ERR_BAD_ARG;  // literals are extracted by the host entry points
  if (len < 0) return TT_ERR_BAD_ARG;
  if (len > TT_MAX_BYTES) return TT_ERR_TOO_LARGE;
  *out_n = 0;
  if (len == 0) return TT_OK;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (hipSetDevice(h->device) != hipSuccess) return TT_ERR_HIP;
  Workspace* s = nullptr;
  int rc = get_ws(h, st, (uint64_t)len, &s);
  if (rc) return rc;
  if (hipMemcpyAsync(s->d_in, utf8, (size_t)len, hipMemcpyHostToDevice, st) != hipSuccess) return TT_ERR_HIP;
  rc = run_chain(h, s, s->d_in, (uint32_t)len, nullptr, 0, s->d_out, s->d_len, nullptr, st, 0);
  if (rc) return rc;
  if (hipMemcpyAsync(s->h_len, s->d_len, 8, hipMemcpyDeviceToHost, st) != hipSuccess) return TT_ERR_HIP;
  if (hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
  const int64_t P = *s->h_len;
  if (P < 0) return (int)P;
  if (P > len) return TT_ERR_HIP;  // cannot happen: at most one piece per byte
  std::vector<uint32_t> tmp((size_t)P);
  if (P > 0) {
    if (hipMemcpyAsync(tmp.data(), s->d_out, 4 * (size_t)P, hipMemcpyDeviceToHost, st) != hipSuccess)
      return TT_ERR_HIP;
    if (hipStreamSynchronize(st) != hipSuccess) return TT_ERR_HIP;
  }
  for (int64_t i = 0; i < P; ++i) out_piece_starts[i] = tmp[(size_t)i];
  *out_n = P;
  return TT_OK;
}

int tt_set_profiling(tt_tokenizer* h, int32_t n_calls) {
  if (!h) return TT_ERR_NULL_ARG;
  if (n_calls < 0 || n_calls > 65536) return TT_ERR_BAD_ARG;
  std::lock_guard<std::mutex> g(h->mu);
  h->profile = n_calls;
  return TT_OK;
}

int tt_stage_times(tt_tokenizer* h, void* stream, double* out_ms, int32_t cap, int32_t* n_out) {
  if (!h || !n_out || (cap > 0 && !out_ms)) return TT_ERR_NULL_ARG;
  *n_out = 0;
  hipStream_t st = static_cast<hipStream_t>(stream);
  Workspace* s = nullptr;
  {
    std::lock_guard<std::mutex> g(h->mu);
    auto it = h->ws.find(st);
    if (it == h->ws.end()) return TT_OK;
    s = it->second;
  }
  if (s->ring == 0 || s->n_calls == 0) return TT_OK;
  if (hipSetDevice(h->device) != hipSuccess) return TT_ERR_HIP;
  const int64_t kept = s->n_calls < s->ring ? s->n_calls : s->ring;
  int k = 0;
  for (int64_t c = s->n_calls - kept; c < s->n_calls && k + N_STAGES <= cap; ++c) {
    hipEvent_t* e = &s->ev[(size_t)(c % s->ring) * (N_STAGES + 1)];
    if (hipEventSynchronize(e[N_STAGES]) != hipSuccess) return TT_ERR_HIP;
    for (int i = 0; i < N_STAGES; ++i) {
      float ms = 0.f;
      if (hipEventElapsedTime(&ms, e[i], e[i + 1]) != hipSuccess) return TT_ERR_HIP;
      out_ms[k++] = ms;
    }
  }
  *n_out = k;
  return TT_OK;
}

}  // extern "C"
