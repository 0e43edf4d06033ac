// Drives the host planner (bucket_plan, epoch_schedule[_ordered]) over random
// and edge-case inputs for a build with AddressSanitizer and
// UndefinedBehaviorSanitizer, checking the invariants the header states.
// Exit status 0 = every check held (the sanitizers abort on their own).
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <vector>

#include "rnnbkt.h"

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint64_t next_u64() {  // splitmix64
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
int rand_int(int lo, int hi) { return lo + (int)(next_u64() % (uint64_t)(hi - lo + 1)); }

int g_fail = 0;
#define CHECK(c)                                                     \
  do {                                                               \
    if (!(c)) {                                                      \
      std::fprintf(stderr, "check failed line %d: %s\n", __LINE__, #c); \
      ++g_fail;                                                      \
    }                                                                \
  } while (0)

std::vector<int32_t> draw_lengths(int law, int n) {
  std::vector<int32_t> v(n);
  for (int i = 0; i < n; ++i) {
    switch (law) {
      case 0: v[i] = rand_int(1, 6); break;                  // many ties
      case 1: v[i] = rand_int(1, 4000); break;               // wide
      case 2: v[i] = 37; break;                               // all equal
      case 3: {                                               // heavy tail
        const double u = (double)(next_u64() >> 11) / 9007199254740992.0;
        v[i] = (int32_t)std::min(4000.0, std::floor(20.0 / std::pow(1.0 - u, 1.0 / 1.5)));
        break;
      }
      default: v[i] = 1 + (int32_t)(next_u64() % 300);
    }
  }
  return v;
}

void check_case(const std::vector<int32_t>& len, int K, int B) {
  const int64_t n = (int64_t)len.size();
  std::vector<int32_t> upper(std::max(K, 1)), bof(n);
  int32_t keff = 0;
  int64_t padded = 0;
  CHECK(rnnbkt_bucket_plan(len.data(), n, K, upper.data(), bof.data(), &keff, &padded) == 0);
  std::vector<int32_t> sorted(len);
  std::sort(sorted.begin(), sorted.end());
  const int distinct = (int)(std::unique(sorted.begin(), sorted.end()) - sorted.begin());
  CHECK(keff == std::min(K, distinct));
  int64_t sum = 0;
  for (int64_t i = 0; i < n; ++i) {
    CHECK(bof[i] >= 0 && bof[i] < keff);
    if (bof[i] < 0 || bof[i] >= keff) return;
    CHECK(len[i] <= upper[bof[i]]);
    CHECK(bof[i] == 0 || len[i] > upper[bof[i] - 1]);
    sum += upper[bof[i]];
  }
  for (int b = 1; b < keff; ++b) CHECK(upper[b - 1] < upper[b]);
  CHECK(sum == padded);
  std::vector<uint64_t> keys(n), okeys(n);
  for (auto& k : keys) k = next_u64();
  for (auto& k : okeys) k = next_u64();
  for (int ordering = 0; ordering < 4; ++ordering) {
    std::vector<int64_t> order(n, -1), start(n + 1, -1);
    int64_t nb = -1;
    CHECK(rnnbkt_epoch_schedule_ordered(len.data(), bof.data(), n, keff, keys.data(), B, ordering,
                                        okeys.data(), order.data(), start.data(), &nb) == 0);
    CHECK(nb >= 1 && nb <= n);
    if (nb < 1 || nb > n) return;
    CHECK(start[0] == 0 && start[nb] == n);
    std::vector<char> seen(n, 0);
    for (int64_t q = 0; q < nb; ++q) {
      const int64_t a = start[q], e = start[q + 1];
      CHECK(a < e && e - a <= B);
      if (!(a < e && e <= n)) return;
      for (int64_t i = a; i < e; ++i) {
        const int64_t s = order[i];
        CHECK(s >= 0 && s < n);
        if (s < 0 || s >= n) return;
        CHECK(!seen[s]);
        seen[s] = 1;
        CHECK(bof[s] == bof[order[a]]);
        if (i > a) CHECK(len[order[i - 1]] >= len[s]);
      }
    }
  }
}

}  // namespace

int main() {
  for (int it = 0; it < 400; ++it) {
    const int n = it < 20 ? 1 + it % 3 : rand_int(1, 3000);
    const auto len = draw_lengths(it % 5, n);
    check_case(len, rand_int(1, 40), rand_int(1, 130));
  }
  // invalid arguments: every call returns an error code and touches nothing else
  int32_t one = 5, zero = 0, keff = 0;
  int32_t up[4], bo[4];
  int64_t pad = 0, ord[4], st[5], nb = 0;
  uint64_t key[4] = {1, 2, 3, 4};
  CHECK(rnnbkt_bucket_plan(nullptr, 1, 1, up, bo, &keff, &pad) < 0);
  CHECK(rnnbkt_bucket_plan(&one, 0, 1, up, bo, &keff, &pad) < 0);
  CHECK(rnnbkt_bucket_plan(&one, 1, 0, up, bo, &keff, &pad) < 0);
  CHECK(rnnbkt_bucket_plan(&zero, 1, 1, up, bo, &keff, &pad) < 0);
  int32_t bof0 = 0, bof_bad = 3;
  CHECK(rnnbkt_epoch_schedule(&one, &bof0, 1, 1, key, 0, ord, st, &nb) < 0);
  CHECK(rnnbkt_epoch_schedule(&one, &bof_bad, 1, 1, key, 1, ord, st, &nb) < 0);
  CHECK(rnnbkt_epoch_schedule_ordered(&one, &bof0, 1, 1, key, 1, 9, key, ord, st, &nb) < 0);
  CHECK(rnnbkt_epoch_schedule_ordered(&one, &bof0, 1, 1, key, 1, RNNBKT_ORDER_RANDOM_BUCKETS,
                                      nullptr, ord, st, &nb) < 0);
  CHECK(rnnbkt_last_error()[0] != '\0');
  std::printf("plan driver: %s\n", g_fail ? "FAILED" : "ok");
  return g_fail ? 1 : 0;
}
