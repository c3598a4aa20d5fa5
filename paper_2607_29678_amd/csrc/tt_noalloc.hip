// tt_encode_device_noalloc: the device entry point for callers that cannot
// allocate (code under stream capture, tight serving loops, hosts that forbid
// allocation during serving).  Its workspace is a file-scope device array of
// fixed size instead of a per-stream allocation; everything else is the same
// chain as tt_encode_device (the same tile kernel, the same placement).
//
// The array's name is a host-side stand-in in host code, not a device
// address: the address is taken once per device, with that device current,
// through hipGetSymbolAddress, and only that address is used afterwards.
// Every call on a device uses that device's one array, which keeps the words
// of the last call: its epoch-tagged tile words are cleared by a fill kernel
// when the array is first set up on the device (and when the 31-bit epoch
// wraps), and each call takes a new epoch, so stale words are never taken for
// fresh ones.  Calls that overlap on one device race for the array.
#include <mutex>

#include "tt_internal.h"

namespace tt {
namespace {

constexpr uint64_t NA_MAX = TT_NOALLOC_MAX_BYTES;
constexpr uint64_t NA_TILES = (NA_MAX + PT_OWN - 1) / PT_OWN + 1;
constexpr uint64_t align256(uint64_t x) { return (x + 255) / 256 * 256; }
// layout: control word, four arrays of epoch-tagged tile words (cleared at
// set-up), staging of incoming units (4 B per byte), rows of long units
// (4 words per byte, then the selection masks)
constexpr uint64_t NA_CTRL = 0;
constexpr uint64_t NA_TSUM = NA_CTRL + align256(sizeof(Ctrl));
constexpr uint64_t NA_TEND = NA_TSUM + align256(8 * NA_TILES);
constexpr uint64_t NA_TLAST = NA_TEND + align256(8 * NA_TILES);
constexpr uint64_t NA_TAGG = NA_TLAST + align256(8 * NA_TILES);
constexpr uint64_t NA_CLEAR = NA_TAGG + align256(8 * NA_TILES);  // bytes cleared at set-up
constexpr uint64_t NA_STAGE = NA_CLEAR;
constexpr uint64_t NA_ROWS = NA_STAGE + align256(4 * NA_MAX);
constexpr uint64_t NA_BYTES = NA_ROWS + align256(16 * NA_MAX + 8 * (NA_MAX / 16 + 8));

static __device__ __align__(256) uint8_t noalloc_scratch[NA_BYTES];

constexpr int MAX_DEVICES = 64;

// Per-device state: the array's device address and the call numbering.
struct DevState {
  std::mutex mu;
  uint8_t* base = nullptr;  // device address of noalloc_scratch on this device
  uint32_t epoch = 0;       // epoch of the latest call (0: the words need clearing)
  uint32_t ticket_base = 0;
};
DevState g_dev[MAX_DEVICES];

__global__ void clear_words(uint64_t* p, uint64_t n_words) {
  for (uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_words; i += (uint64_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

__global__ void set_len(int64_t* p, int64_t v) {
  if (threadIdx.x == 0 && blockIdx.x == 0) *p = v;
}

}  // namespace
}  // namespace tt

using namespace tt;

extern "C" int tt_encode_device_noalloc(tt_tokenizer* h, const uint8_t* d_utf8, int64_t len, int32_t* d_out_ids,
                                        int64_t* d_out_len, void* stream) {
  if (!h || !d_out_len || (len > 0 && (!d_utf8 || !d_out_ids))) return TT_ERR_NULL_ARG;
  if (handle_has_added(h)) return TT_ERR_BAD_ARG;  // literals are extracted by the host entry points
  if (len < 0) return TT_ERR_BAD_ARG;
  if ((uint64_t)len > NA_MAX) return TT_ERR_TOO_LARGE;
  const int dev = handle_device(h);
  if (dev < 0 || dev >= MAX_DEVICES) return TT_ERR_BAD_ARG;
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (hipSetDevice(dev) != hipSuccess) return TT_ERR_HIP;
  if (len == 0) {
    hipLaunchKernelGGL(set_len, dim3(1), dim3(64), 0, st, d_out_len, (int64_t)0);
    return hipGetLastError() == hipSuccess ? TT_OK : TT_ERR_HIP;
  }
  DevState& ds = g_dev[dev];
  std::lock_guard<std::mutex> g(ds.mu);
  if (ds.base == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(noalloc_scratch)) != hipSuccess || p == nullptr) return TT_ERR_HIP;
    ds.base = static_cast<uint8_t*>(p);
    ds.epoch = 0;
  }
  if (ds.epoch == 0 || ds.epoch + 1 >= EPOCH_LIMIT) {
    // first call on this device, or the epochs wrapped: clear the words that
    // carry them (a kernel, not a memset, so that the call may be captured)
    hipLaunchKernelGGL(clear_words, dim3(64), dim3(256), 0, st, reinterpret_cast<uint64_t*>(ds.base), NA_CLEAR / 8);
    if (hipGetLastError() != hipSuccess) return TT_ERR_HIP;
    ds.epoch = 0;
    ds.ticket_base = 0;
  }
  uint8_t* b = ds.base;
  Work w{};
  w.text = d_utf8;
  w.n = (uint32_t)len;
  w.doc_off = nullptr;
  w.n_docs = 0;
  w.ctrl = reinterpret_cast<Ctrl*>(b + NA_CTRL);
  w.epoch = ++ds.epoch;
  w.ticket_base = ds.ticket_base;
  w.n_tiles = n_tiles_for((uint32_t)len);
  w.tile_sum = reinterpret_cast<uint64_t*>(b + NA_TSUM);
  w.tile_end = reinterpret_cast<uint64_t*>(b + NA_TEND);
  w.tile_last = reinterpret_cast<uint64_t*>(b + NA_TLAST);
  w.tile_agg = reinterpret_cast<uint64_t*>(b + NA_TAGG);
  w.stage = reinterpret_cast<uint32_t*>(b + NA_STAGE);
  w.scratch = reinterpret_cast<uint32_t*>(b + NA_ROWS);
  w.out_ids = d_out_ids;
  w.out_len = d_out_len;
  const DevTables tb = handle_tables(h);
  if (launch_tile(w, tb, handle_pattern(h), 1, handle_ignore(h), st) != hipSuccess) return TT_ERR_HIP;
  ds.ticket_base += w.n_tiles;  // the tiles took their tickets
  return TT_OK;
}
