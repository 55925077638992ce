// Single-pass decoupled look-back over workgroups (stable compaction across a grid): the
// published method of Merrill and Garland (single-pass prefix scan with decoupled
// look-back, 2016), here in a wave-wide form.
//
// Workgroup k (in ticket order, so every workgroup it waits on has already started)
// publishes its own count as an "aggregate", finds the total of all earlier workgroups by
// reading their state words, and publishes the running total as "inclusive". One 64-bit
// word per workgroup holds the flag (high half) and the count (low half), so a single
// atomic load sees a consistent pair; nothing else is ordered by these words, so relaxed
// device-scope atomics suffice.
//
// The reading is done by a whole wave: lane l looks at workgroup k - 1 - l, a ballot
// finds the nearest inclusive word, and the wave adds the counts up to it, or steps back
// 64 workgroups at a time. Waits are bounded (kLookbackSpin tries, far more than any
// running workgroup needs to publish). A word still unset after that -- a predecessor that
// never ran -- ends the wait: the prefix is then wrong, so the workgroup reports failure
// and publishes its inclusive word with an error bit, which every later workgroup whose
// prefix passes through it inherits; the caller turns it into an error count.
#ifndef TG_LOOKBACK_H
#define TG_LOOKBACK_H

#include <hip/hip_runtime.h>

#include <climits>
#include <cstdint>

namespace tg_detail {

constexpr uint64_t kLookAggregate = uint64_t(1) << 32;
constexpr uint64_t kLookInclusive = uint64_t(2) << 32;
constexpr uint64_t kLookError = uint64_t(4) << 32;  // with kLookInclusive: prefix is wrong
constexpr uint32_t kLookbackSpin = 1u << 22;

__device__ __forceinline__ uint64_t look_load(const uint64_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void look_store(uint64_t *p, uint64_t v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Called by all 64 lanes of one wave of workgroup k (k = its ticket) with the
// workgroup's own count; returns (in every lane) the total count of workgroups 0..k-1
// and publishes this workgroup's inclusive total. *failed (every lane) is true when the
// prefix could not be established (see the header comment).
__device__ __forceinline__ int lookback_prefix(uint64_t *state, int k, int count,
                                               bool *failed) {
  const int lane = threadIdx.x & 63;
  *failed = false;
  if (k == 0) {
    if (lane == 0) look_store(&state[0], kLookInclusive | uint32_t(count));
    return 0;
  }
  if (lane == 0) look_store(&state[k], kLookAggregate | uint32_t(count));
  int prefix = 0;
  bool err = false;
  for (int j = k - 1; j >= 0; j -= 64) {
    const int idx = j - lane;
    uint64_t s = idx >= 0 ? look_load(&state[idx]) : kLookInclusive;
    for (uint32_t spin = 0; __ballot((s >> 32) == 0) != 0 && spin < kLookbackSpin; ++spin)
      if ((s >> 32) == 0) s = look_load(&state[idx]);
    if ((s >> 32) == 0) s = kLookInclusive | kLookError;  // timed out: count unknown
    const uint64_t inc = __ballot((s & kLookInclusive) != 0);
    const int stop = inc ? __builtin_ctzll(inc) : 63;  // nearest inclusive lane, or all
    int v = lane <= stop ? static_cast<int>(static_cast<uint32_t>(s)) : 0;
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    prefix += v;
    err = err || __ballot(lane <= stop && (s & kLookError) != 0) != 0;
    if (inc) break;
  }
  if (lane == 0)
    look_store(&state[k], kLookInclusive | (err ? kLookError : 0) | uint32_t(prefix + count));
  *failed = err;
  return prefix;
}

// Workgroup-wide form, called by every thread of a workgroup of kThreads threads (a
// multiple of 64) with the workgroup's count: each step reads the kThreads * kPer state
// words before the current position at once (kPer per thread), the nearest inclusive
// word among them ends the walk, and the counts up to it are summed over the workgroup.
// A grid of many workgroups reaches an inclusive word in about 1 / (4 kPer) of the steps
// of the one-wave form. Same results, bounds and failure reporting as lookback_prefix.
template <int kThreads, int kPer>
__device__ __forceinline__ int lookback_prefix_block(uint64_t *state, int k, int count,
                                                     bool *failed) {
  constexpr int kWaves = kThreads / 64;
  constexpr int kSpan = kThreads * kPer;
  __shared__ int s_stop[kWaves], s_sum[kWaves], s_err[kWaves];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  *failed = false;
  if (k == 0) {
    if (tid == 0) look_store(&state[0], kLookInclusive | uint32_t(count));
    return 0;
  }
  if (tid == 0) look_store(&state[k], kLookAggregate | uint32_t(count));
  int prefix = 0;
  bool err = false;
  for (int j = k - 1; j >= 0; j -= kSpan) {
    uint64_t s[kPer];
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int idx = j - tid - kThreads * i;
      s[i] = idx >= 0 ? look_load(&state[idx]) : kLookInclusive;
    }
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      const int idx = j - tid - kThreads * i;
      for (uint32_t spin = 0; (s[i] >> 32) == 0 && spin < kLookbackSpin; ++spin)
        s[i] = look_load(&state[idx]);
      if ((s[i] >> 32) == 0) s[i] = kLookInclusive | kLookError;  // timed out: count unknown
    }
    // distance (from j) of the nearest inclusive word, over the workgroup
    int stop = INT_MAX;
#pragma unroll
    for (int i = kPer - 1; i >= 0; --i)
      if (s[i] & kLookInclusive) stop = tid + kThreads * i;
    for (int o = 32; o > 0; o >>= 1) stop = min(stop, __shfl_xor(stop, o));
    if (lane == 0) s_stop[wave] = stop;
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kWaves; ++w) stop = min(stop, s_stop[w]);
    int v = 0, e = 0;
#pragma unroll
    for (int i = 0; i < kPer; ++i) {
      if (tid + kThreads * i > stop) continue;
      v += static_cast<int>(static_cast<uint32_t>(s[i]));
      e |= (s[i] & kLookError) != 0;
    }
    for (int o = 32; o > 0; o >>= 1) {
      v += __shfl_xor(v, o);
      e |= __shfl_xor(e, o);
    }
    if (lane == 0) {
      s_sum[wave] = v;
      s_err[wave] = e;
    }
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      prefix += s_sum[w];
      err = err || s_err[w] != 0;
    }
    if (stop != INT_MAX) break;
  }
  if (tid == 0)
    look_store(&state[k], kLookInclusive | (err ? kLookError : 0) | uint32_t(prefix + count));
  *failed = err;
  return prefix;
}

}  // namespace tg_detail

#endif  // TG_LOOKBACK_H
