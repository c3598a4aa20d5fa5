// Host copies of the staging buffers (tt_copy.cpp), split among a few worker
// threads.  Plain C++ (no HIP), so that the pool can also be built and
// stress-tested on its own.
#pragma once

#include <cstddef>
#include <cstdint>

namespace tt {

// Copy n bytes (the regions must not overlap).  Copies of at least 256 KB are
// split among the calling thread and the pool's workers; smaller ones, and
// copies while another thread's copy is running, are a plain memcpy.
void host_copy(void* dst, const void* src, size_t n);

// dst[i] = lo[i] | hi[i] << 16 for i < count (hi == nullptr: dst[i] = lo[i]),
// IDs staged as 16 or 24 bits widened to int32, split the same way as
// host_copy (by output bytes).
void host_widen(int32_t* dst, const uint16_t* lo, const uint8_t* hi, size_t count);

// Let sleeping workers start spinning ahead of a copy of n bytes (cheap when
// they are awake; nothing for copies too small to be split).
void host_copy_wake(size_t n);

}  // namespace tt
