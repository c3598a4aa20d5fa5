// Span export (the step after compaction): the byte and character span of
// every token.  For byte-level BPE a token's byte length is fixed by the
// vocabulary, so byte offsets are a running sum of token lengths, and a
// running count of the text's non-continuation bytes lifts them to character
// spans (Appendix, Route C, span export; the records of Definition d:records).
//
// The tile kernel has already written every token's byte start and, for every
// 4-byte word of the request, the number of non-continuation bytes before it.
// Here each token gets
//   byte end    = the next token's byte start (the request's length for the last),
//   char begin  = the index of the character holding its first byte,
//   char end    = one past the character holding its last byte,
// so tokens that split one multi-byte character all report that character.
#include "tt_internal.h"

namespace tt {

namespace {

__global__ __launch_bounds__(256) void spans_kernel(Work w) {
  const int64_t T = *w.out_len;  // written by the tile kernel on this stream; < 0 on error
  if (T <= 0) return;
  const uint32_t n = w.n;
  const uint8_t* __restrict__ text = w.text;
  const uint32_t* __restrict__ cc = w.ccount;
  // non-continuation bytes in [0, p), for p <= n (reads bytes below p only)
  auto count_before = [&](uint32_t p) -> uint32_t {
    uint32_t c = cc[p >> 2];
    for (uint32_t q = p & ~3u; q < p; ++q) c += (text[q] & 0xC0u) != 0x80u ? 1u : 0u;
    return c;
  };
  const uint32_t stride = gridDim.x * blockDim.x;
  for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < (uint64_t)T; i += stride) {
    int32_t* r = w.out_spans + 4 * (size_t)i;
    // (valid output has 0 <= begin < end <= n; the bounds only keep reads in range)
    const uint32_t bb = min((uint32_t)r[0], n - 1u);
    const uint32_t be = min(i + 1 < (uint64_t)T ? (uint32_t)w.out_spans[4 * (size_t)(i + 1)] : n, n);
    r[1] = (int32_t)be;
    r[2] = (int32_t)(count_before(bb + 1u) - 1u);
    r[3] = (int32_t)count_before(be);
  }
}

}  // namespace

hipError_t launch_spans(const Work& w, hipStream_t s) {
  // at most one token per byte; the grid covers that bound with a stride loop
  uint32_t blocks = (w.n + 255u) / 256u;
  if (blocks > 2048u) blocks = 2048u;
  if (blocks == 0u) blocks = 1u;
  hipLaunchKernelGGL(spans_kernel, dim3(blocks), dim3(256), 0, s, w);
  return hipGetLastError();
}

}  // namespace tt
