// Host side of the method: optimal length bucketing (Sec. III.A) and the
// per-epoch mini-batch schedule (Sec. III, Sec. IV.A).  Pure integer work.
#include <algorithm>
#include <cstring>
#include <limits>
#include <numeric>
#include <vector>

#include "common.h"

namespace rnnbkt {

namespace {
thread_local std::string g_err;
}

void set_error(const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
}

void clear_error() { g_err.clear(); }

const char* last_error() { return g_err.c_str(); }

}  // namespace rnnbkt

extern "C" const char* rnnbkt_last_error(void) { return rnnbkt::last_error(); }

// The DP of Sec. III.A over the length histogram.  The paper's table is
// indexed by every length 1..Lmax; here it is indexed by the D distinct
// lengths v_0 < ... < v_{D-1} present.  With K <= D buckets every optimal
// split uses only present lengths as upper bounds and has no empty bucket
// (an empty bucket could be traded for splitting a bucket holding two
// distinct lengths, and a bound above the bucket's largest length could be
// lowered, both at strictly lower cost), so the candidate split points of the
// full table that can reach the minimum are exactly the present ones and the
// two tables select the same split points under the same tie rule.
//   dp[q][i] = min_{0 <= j < i} dp[q-1][j] + v_{i-1} * (F[i] - F[j])
// with F[i] = number of sequences whose length is among v_0..v_{i-1};
// j is scanned downwards and only a strictly smaller score replaces the
// incumbent (largest minimising j wins).
extern "C" int32_t rnnbkt_bucket_plan(const int32_t* lengths, int64_t n, int32_t K,
                                      int32_t* bucket_upper, int32_t* bucket_of,
                                      int32_t* K_eff, int64_t* padded_steps) {
  using rnnbkt::clear_error;
  clear_error();
  RNNBKT_REQUIRE(lengths && bucket_upper && bucket_of && K_eff && padded_steps,
                 RNNBKT_EINVAL, "bucket_plan: null pointer");
  RNNBKT_REQUIRE(n >= 1, RNNBKT_EINVAL, "bucket_plan: n must be >= 1 (got %lld)", (long long)n);
  RNNBKT_REQUIRE(K >= 1, RNNBKT_EINVAL, "bucket_plan: K must be >= 1 (got %d)", K);
  for (int64_t s = 0; s < n; ++s)
    RNNBKT_REQUIRE(lengths[s] >= 1, RNNBKT_EINVAL,
                   "bucket_plan: lengths[%lld] = %d < 1", (long long)s, lengths[s]);
  // Length histogram f (Sec. III.A) restricted to the distinct lengths, from
  // a sorted copy: O(n) memory whatever the largest length is.
  std::vector<int32_t> sorted(lengths, lengths + n);
  std::sort(sorted.begin(), sorted.end());
  std::vector<int64_t> v, F(1, 0);
  for (int64_t s = 0; s < n;) {
    int64_t e = s + 1;
    while (e < n && sorted[e] == sorted[s]) ++e;
    v.push_back(sorted[s]);
    F.push_back(F.back() + (e - s));
    s = e;
  }
  const int D = static_cast<int>(v.size());
  const int Q = std::min<int>(K, D);
  const int64_t INF = std::numeric_limits<int64_t>::max() / 4;
  std::vector<int64_t> prev_row(D + 1, INF), cur_row(D + 1, INF);
  std::vector<int32_t> arg(static_cast<size_t>(Q + 1) * (D + 1), -1);
  prev_row[0] = 0;  // dp[0][0] = 0, dp[0][i>0] = INF
  for (int q = 1; q <= Q; ++q) {
    std::fill(cur_row.begin(), cur_row.end(), INF);
    for (int i = 1; i <= D; ++i) {
      const int64_t up = v[i - 1];
      int64_t best = INF;
      int32_t bj = -1;
      for (int j = i - 1; j >= 0; --j) {
        if (prev_row[j] == INF) continue;
        const int64_t val = up * (F[i] - F[j]) + prev_row[j];
        if (val < best) {
          best = val;
          bj = j;
        }
      }
      cur_row[i] = best;
      arg[static_cast<size_t>(q) * (D + 1) + i] = bj;
    }
    std::swap(prev_row, cur_row);
  }
  // Backtrack from the full set (i = D) through Q levels.
  int i = D;
  for (int q = Q; q >= 1; --q) {
    bucket_upper[q - 1] = static_cast<int32_t>(v[i - 1]);
    i = arg[static_cast<size_t>(q) * (D + 1) + i];
  }
  int64_t padded = 0;
  std::vector<int64_t> counts(Q, 0);
  for (int64_t s = 0; s < n; ++s) {
    const int32_t* p = std::lower_bound(bucket_upper, bucket_upper + Q, lengths[s]);
    const int32_t b = static_cast<int32_t>(p - bucket_upper);
    bucket_of[s] = b;
    counts[b]++;
  }
  for (int b = 0; b < Q; ++b) padded += counts[b] * static_cast<int64_t>(bucket_upper[b]);
  *K_eff = Q;
  *padded_steps = padded;
  return RNNBKT_OK;
}

extern "C" int32_t rnnbkt_epoch_schedule_ordered(const int32_t* lengths,
                                                 const int32_t* bucket_of, int64_t n,
                                                 int32_t K_eff, const uint64_t* keys,
                                                 int32_t B, int32_t ordering,
                                                 const uint64_t* order_keys, int64_t* order,
                                                 int64_t* batch_start, int64_t* num_batches) {
  rnnbkt::clear_error();
  RNNBKT_REQUIRE(lengths && bucket_of && keys && order && batch_start && num_batches,
                 RNNBKT_EINVAL, "epoch_schedule: null pointer");
  RNNBKT_REQUIRE(n >= 1 && K_eff >= 1 && B >= 1, RNNBKT_EINVAL,
                 "epoch_schedule: need n >= 1, K_eff >= 1, B >= 1");
  RNNBKT_REQUIRE(ordering >= RNNBKT_ORDER_ASCENDING && ordering <= RNNBKT_ORDER_SHUFFLED_BATCHES,
                 RNNBKT_EINVAL, "epoch_schedule: unknown ordering %d", ordering);
  const bool keyed =
      ordering == RNNBKT_ORDER_RANDOM_BUCKETS || ordering == RNNBKT_ORDER_SHUFFLED_BATCHES;
  RNNBKT_REQUIRE(!keyed || order_keys, RNNBKT_EINVAL,
                 "epoch_schedule: this ordering needs order_keys");
  RNNBKT_REQUIRE(ordering != RNNBKT_ORDER_RANDOM_BUCKETS || K_eff <= n, RNNBKT_EINVAL,
                 "epoch_schedule: K_eff %d > n leaves buckets without a key", K_eff);
  std::vector<std::vector<int64_t>> members(K_eff);
  for (int64_t s = 0; s < n; ++s) {
    RNNBKT_REQUIRE(bucket_of[s] >= 0 && bucket_of[s] < K_eff, RNNBKT_EINVAL,
                   "epoch_schedule: bucket_of[%lld] = %d outside [0, %d)", (long long)s,
                   bucket_of[s], K_eff);
    RNNBKT_REQUIRE(lengths[s] >= 1, RNNBKT_EINVAL, "epoch_schedule: length < 1");
    members[bucket_of[s]].push_back(s);
  }
  // Bucket order: ascending, descending, or by (order_keys[b], b).
  std::vector<int32_t> bucket_seq(K_eff);
  for (int32_t b = 0; b < K_eff; ++b)
    bucket_seq[b] = ordering == RNNBKT_ORDER_DESCENDING ? K_eff - 1 - b : b;
  if (ordering == RNNBKT_ORDER_RANDOM_BUCKETS)
    std::sort(bucket_seq.begin(), bucket_seq.end(), [&](int32_t a, int32_t c) {
      return order_keys[a] != order_keys[c] ? order_keys[a] < order_keys[c] : a < c;
    });
  // Batches are built in the bucket sequence; each is written as a contiguous
  // run of `order` and recorded by its [begin, end) range.
  std::vector<int64_t> ranges;  // begin of batch i at 2i, end at 2i+1
  std::vector<int64_t> staged(static_cast<size_t>(n));
  int64_t pos = 0;
  for (int32_t b : bucket_seq) {
    auto& m = members[b];
    std::sort(m.begin(), m.end(), [&](int64_t a, int64_t c) {
      return keys[a] != keys[c] ? keys[a] < keys[c] : a < c;
    });
    for (size_t st = 0; st < m.size(); st += B) {
      const size_t en = std::min(m.size(), st + static_cast<size_t>(B));
      std::sort(m.begin() + st, m.begin() + en, [&](int64_t a, int64_t c) {
        return lengths[a] != lengths[c] ? lengths[a] > lengths[c] : a < c;
      });
      ranges.push_back(pos);
      for (size_t k = st; k < en; ++k) staged[pos++] = m[k];
      ranges.push_back(pos);
    }
  }
  const int64_t nb = static_cast<int64_t>(ranges.size() / 2);
  // Batch order: as built, or by (order_keys[i], i) with i the batch's
  // position in the ascending build (the bucket sequence is ascending here).
  std::vector<int64_t> batch_seq(nb);
  for (int64_t i = 0; i < nb; ++i) batch_seq[i] = i;
  if (ordering == RNNBKT_ORDER_SHUFFLED_BATCHES)
    std::sort(batch_seq.begin(), batch_seq.end(), [&](int64_t a, int64_t c) {
      return order_keys[a] != order_keys[c] ? order_keys[a] < order_keys[c] : a < c;
    });
  pos = 0;
  batch_start[0] = 0;
  for (int64_t i = 0; i < nb; ++i) {
    const int64_t j = batch_seq[i];
    for (int64_t k = ranges[2 * j]; k < ranges[2 * j + 1]; ++k) order[pos++] = staged[k];
    batch_start[i + 1] = pos;
  }
  *num_batches = nb;
  return RNNBKT_OK;
}

extern "C" int32_t rnnbkt_epoch_schedule(const int32_t* lengths, const int32_t* bucket_of,
                                         int64_t n, int32_t K_eff, const uint64_t* keys,
                                         int32_t B, int64_t* order, int64_t* batch_start,
                                         int64_t* num_batches) {
  return rnnbkt_epoch_schedule_ordered(lengths, bucket_of, n, K_eff, keys, B,
                                       RNNBKT_ORDER_ASCENDING, nullptr, order, batch_start,
                                       num_batches);
}
