// Host-only exercise of the library's argument checks and plan building under
// AddressSanitizer (host-side instrumentation only; nothing here touches a GPU):
// random segment tables, some corrupted on purpose, through the size queries of
// the attention step, the offline producer and the protected-set construction,
// and NULL / out-of-range arguments on the other entry points.
#include <cstdio>
#include <cstdint>
#include <cstdlib>
#include <vector>
#include <random>
#include <algorithm>
#include <numeric>
#include "mla_online.h"
int main() {
  std::mt19937_64 rng(7);
  int ok = 0, rejected = 0;
  for (int it = 0; it < 3000; ++it) {
    const int nd = 1 + rng() % 12;
    std::vector<int64_t> len(nd);
    for (auto& l : len) l = 1 + rng() % 400;
    const int tq = rng() % 50;
    std::vector<int> perm(nd);
    std::iota(perm.begin(), perm.end(), 0);
    std::shuffle(perm.begin(), perm.end(), rng);
    std::vector<mla_segment> segs;
    int64_t ks = 0;
    std::vector<int64_t> req(nd);
    int64_t acc = 0;
    for (int d : perm) { req[d] = acc; acc += len[d]; }
    for (int d = 0; d < nd; ++d) { segs.push_back({ks, len[d], req[d]}); ks += len[d]; }
    if (tq) segs.push_back({ks, tq, acc});
    const int64_t N = ks + tq;
    // occasionally corrupt the table
    const int corrupt = rng() % 10;
    if (corrupt == 0) segs[rng() % segs.size()].length = 0;
    if (corrupt == 1) segs[rng() % segs.size()].req_offset += 1;
    if (corrupt == 2) segs[rng() % segs.size()].kv_start = -1;
    std::vector<int32_t> prot;
    for (int64_t r = 0; r < N; ++r) if (rng() % 7 == 0) prot.push_back((int32_t)r);
    if (corrupt == 3 && !prot.empty()) prot.push_back(prot.front());
    const int G = 1 << (rng() % 3), hpg = 1 + rng() % 4;
    mla_geom g{G * hpg, G, 512, 64, 64 * G, G, 0.07f, 10000.0, (int32_t)(rng() % 2)};
    int64_t n_slots = 0, n_parts = 0;
    size_t ws = 0;
    const int64_t split = (rng() % 3 == 0) ? 0 : (int64_t)(rng() % 500);
    mla_status s = mla_online_attend_query(&g, segs.data(), (int32_t)segs.size(), prot.data(), (int32_t)prot.size(),
                                           split, &n_slots, &n_parts, &ws);
    size_t w2 = 0, w3 = 0;
    mla_status s2 = mla_offline_produce_query(&g, segs.data(), (int32_t)segs.size(), &w2);
    mla_status s3 = mla_protected_rows_query(segs.data(), (int32_t)segs.size(), &w3);
    if (s == MLA_OK) ++ok; else ++rejected;
    if ((corrupt == 0 || corrupt == 2 || corrupt == 3) && s == MLA_OK) {
      printf("corrupted table %d accepted\n", corrupt);
      return 1;
    }
    if (corrupt > 3 && s != MLA_OK) {
      printf("valid table rejected: %s\n", mla_last_error_detail());
      return 1;
    }
    (void)s2; (void)s3;
  }
  // invalid arguments on every entry point that validates before touching the GPU
  mla_geom g{8, 2, 512, 64, 128, 2, 0.07f, 10000.0, 0};
  mla_segment seg{0, 10, 0};
  printf("null checks: %d %d %d %d\n", mla_online_attend_query(nullptr, &seg, 1, nullptr, 0, 0, nullptr, nullptr, nullptr),
         mla_segment_merge(-1, 512, nullptr, nullptr, nullptr, 0, nullptr, nullptr, nullptr),
         mla_moe_fanout(4, 16, nullptr, 6, 3, 0.9f, nullptr, nullptr, nullptr, nullptr, nullptr),
         mla_shared_wb(4, 64, 16, nullptr, nullptr, 1, nullptr, nullptr));
  printf("random tables: %d accepted, %d rejected\n", ok, rejected);
  return 0;
}
