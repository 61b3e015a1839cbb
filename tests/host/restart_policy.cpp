// CPU check of the attention kernel's restart policy (restart.h): which weight
// sums vote, how far they raise the reference, and that a work item's passes
// are bounded.  Built with hipcc as host code only; no GPU call is made.
#include <cfloat>
#include <cmath>
#include <cstdio>

#include "restart.h"

using namespace mla;

static int fails = 0;
#define CHECK(cond)                                                  \
  do {                                                               \
    if (!(cond)) {                                                   \
      std::printf("FAIL line %d: %s\n", __LINE__, #cond);            \
      ++fails;                                                       \
    }                                                                \
  } while (0)

// passes the kernel makes over an item with one head-row whose tile weights sum
// to 2^(peak - m_run) against the reference m_run (fp32, overflow to +inf), when
// the item's first tile set m_run = first
static int passes(float first, float peak) {
  float m_run = first, m_seen = first;
  for (int attempt = 0;; ++attempt) {
    const float rsum = std::exp2f(peak - m_run);
    if (restart_allowed(attempt) && restart_vote(rsum)) {
      const float r = restart_raise(rsum);
      m_seen = raised_reference(m_seen, m_run, r, r);
      m_run = m_seen;
      continue;
    }
    return attempt + 1;
  }
}

int main() {
  const float two64 = 0x1p64f;
  // votes
  CHECK(!restart_vote(NAN));
  CHECK(!restart_vote(-NAN));
  CHECK(restart_vote(INFINITY));
  CHECK(!restart_vote(-INFINITY));
  CHECK(!restart_vote(0.f));
  CHECK(!restart_vote(1.f));
  CHECK(restart_vote(two64));
  CHECK(!restart_vote(std::nextafterf(two64, 0.f)));
  CHECK(restart_vote(std::nextafterf(two64, INFINITY)));
  CHECK(restart_vote(FLT_MAX));
  // raises
  CHECK(restart_raise(two64) == 64.f);
  CHECK(restart_raise(0x1p70f) == 70.f);
  CHECK(restart_raise(INFINITY) == 128.f);
  CHECK(restart_raise(NAN) == -INFINITY);                       // no vote: no raise
  CHECK(restart_raise(1.f) == -INFINITY);
  CHECK(restart_raise(std::nextafterf(two64, 0.f)) == -INFINITY);
  // attempts
  CHECK(kMaxAttempts == 16);
  for (int a = 0; a + 1 < kMaxAttempts; ++a) CHECK(restart_allowed(a));
  CHECK(!restart_allowed(kMaxAttempts - 1));
  CHECK(!restart_allowed(kMaxAttempts));
  // the next reference
  CHECK(raised_reference(-1e30f, 5.f, 64.f, 10.f) == 69.f);
  CHECK(raised_reference(80.f, 5.f, 64.f, 10.f) == 80.f);
  CHECK(raised_reference(7.f, 5.f, restart_raise(NAN), restart_raise(NAN)) == 7.f);   // a NaN sum raises nothing
  CHECK(raised_reference(7.f, 5.f, restart_raise(NAN), 70.f) == 75.f);                 // its lane partner still does
  CHECK(raised_reference(5.f, 5.f, restart_raise(3.f), restart_raise(1e18f)) == 5.f);   // no vote: unchanged
  CHECK(std::isinf(raised_reference(-1e30f, INFINITY, 64.f, 64.f)));
  CHECK(raised_reference(1e38f, 1e38f, 128.f, 128.f) == 1e38f);   // a raise lost to rounding
  // bounded passes
  CHECK(passes(0.f, 10.f) == 1);          // within range: no restart
  CHECK(passes(0.f, 64.f) == 2);          // sum 2^64 exactly: one restart
  CHECK(passes(0.f, 63.9f) == 1);
  CHECK(passes(0.f, 100.f) == 2);         // raised by log2(2^100): exact
  CHECK(passes(0.f, 288.5f) == 3);        // +200 nats: overflow (+128), then finite
  CHECK(passes(0.f, 1000.f) == 9);        // seven overflow raises of 128, one of log2(2^104), done
  CHECK(passes(0.f, 3000.f) == kMaxAttempts);   // more than 15 raises of 128 would be needed
  CHECK(passes(0.f, INFINITY) == kMaxAttempts); // an infinite score: bounded, then NaN
  CHECK(passes(1e38f, 1e38f * 2.f) == kMaxAttempts);   // raises lost to rounding: bounded
  CHECK(passes(NAN, 5.f) == 1);           // a NaN reference: NaN weights, no vote
  CHECK(passes(0.f, NAN) == 1);           // a NaN score: no vote
  std::printf("restart policy: %d failure(s)\n", fails);
  return fails == 0 ? 0 : 1;
}
