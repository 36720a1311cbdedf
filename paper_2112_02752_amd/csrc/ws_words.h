// Arithmetic of the workspace's call generations, of the tagged words the
// dedup's workgroups publish to one another, and of the per-call error word.
// Plain integer code, compiled into the kernels and, by the CPU tests, with a
// host compiler on its own.
#pragma once

#include <stdint.h>

#if defined(__HIPCC__)
#define EMB_HD __host__ __device__
#else
#define EMB_HD
#endif

namespace emb {

// Generation of the call after one of generation g.  Zero never occurs (a
// cleared word carries generation 0), so generations repeat with period
// 2^32 - 1 calls.
EMB_HD constexpr uint32_t next_gen(uint32_t g) { return g == 0xffffffffu ? 1u : g + 1u; }

// A published word holds a count or offset below 2^30 (a batch has fewer
// than 2^30 ids) in bits 0-29, the sort pass in bits 30-31 and the call's
// generation in bits 32-63.
constexpr uint64_t kWordCountMask = (1ull << 30) - 1ull;

EMB_HD constexpr uint64_t word_tag(uint32_t g, uint32_t pass) {
  return ((uint64_t)g << 32) | ((uint64_t)(pass & 3u) << 30);
}
EMB_HD constexpr uint64_t word_make(uint64_t tag, uint32_t count) { return tag | ((uint64_t)count & kWordCountMask); }
// whether word w was published under `tag` (the same call and pass)
EMB_HD constexpr bool word_current(uint64_t w, uint64_t tag) { return (w & ~kWordCountMask) == tag; }
EMB_HD constexpr uint32_t word_count(uint64_t w) { return (uint32_t)(w & kWordCountMask); }

// Error word: (generation << 32) | error bits of the last call that set any.
// The bits of call g (0 if the word belongs to another call):
EMB_HD constexpr uint32_t err_bits_of(uint64_t w, uint32_t g) { return (uint32_t)(w >> 32) == g ? (uint32_t)w : 0u; }
// the word after call g sets `bits`: added to g's bits, or replacing another call's
EMB_HD constexpr uint64_t err_word_with(uint64_t w, uint32_t g, uint32_t bits) {
  return (uint32_t)(w >> 32) == g ? (w | bits) : (((uint64_t)g << 32) | bits);
}

}  // namespace emb
