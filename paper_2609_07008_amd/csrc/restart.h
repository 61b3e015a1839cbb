// Restart policy of the attention tile loop (Alg. 2 SelectiveMLA with the
// stable log-sum-exp of SegmentedLSEMerge).
//
// The tile loop scales every weight against a fixed reference max m_run (log2
// units), set from an item's first tile, so a later tile's weights 2^(s - m_run)
// are not bounded by 1.  A lane whose weights in one tile sum to 2^64 or more
// (finite or +inf) votes to restart the work item with a raised reference; fp32
// sums and bf16 weights below 2^64 hold every weight without loss.  The rules
// below are shared by the kernel and a CPU test:
//   - only a sum >= 2^64 votes; NaN never does (a NaN score, key or query makes
//     its head-row NaN, which no reference can repair);
//   - the raise is log2 of the sum (at least 64), or 128 when a weight or the
//     sum overflowed fp32; a head-row whose two lanes cast no vote keeps its
//     reference, so a restart recomputes it bit for bit;
//   - an item makes at most kMaxAttempts passes: the last one casts no vote, so
//     the loop ends even when a raise cannot help (an infinite score, or a
//     reference so large that adding 128 does not change it).  Weights that
//     still overflow then give inf / inf = NaN in that head-row's output, as
//     IEEE arithmetic does.  Each pass ends at the first tile where some
//     head-row votes, so finite inputs reach the cap only when an item's
//     head-rows need raises at more than 15 distinct tiles; a head-row left
//     below its ideal reference is still exact while its weights stay below
//     the fp32 range (2^128).
#pragma once

#include <hip/hip_runtime.h>

#include <cmath>

namespace mla {

constexpr float kRestartSum = 0x1p64f;    // a lane's tile weight sum at or above this votes
constexpr float kOverflowRaise = 128.f;   // raise (log2 units) after an fp32 overflow
constexpr int kMaxAttempts = 16;          // passes over one work item: at most 15 restarts

// does this lane's tile weight sum ask for a higher reference?
__host__ __device__ inline bool restart_vote(float rsum) { return rsum >= kRestartSum; }

// how far (log2 units) the lane asks to raise its reference: -inf when it casts
// no vote, so that a restart leaves the reference of every head-row that did not
// ask for it unchanged (those head-rows are then recomputed bit for bit)
__host__ __device__ inline float restart_raise(float rsum) {
  if (!restart_vote(rsum)) return -INFINITY;
  return rsum >= INFINITY ? kOverflowRaise : log2f(rsum);
}

// may pass `attempt` (0-based) of a work item still vote?
__host__ __device__ inline bool restart_allowed(int attempt) { return attempt + 1 < kMaxAttempts; }

// reference of a head-row for the next pass: the largest of what it has seen so
// far and its current reference plus the larger raise of its two lane halves
__host__ __device__ inline float raised_reference(float m_seen, float m_run, float raise_a, float raise_b) {
  return fmaxf(m_seen, m_run + fmaxf(raise_a, raise_b));
}

}  // namespace mla
