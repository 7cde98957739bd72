// Variance-Reduced Sequence Placement (Sec. 4.2 of the Libra paper,
// Algorithm 1): pools of exactly P packed sequences formed from one
// optimizer-step window by exact-cardinality longest-processing-time-first
// placement on the workload F = sum of squared sample lengths (Eq. 4).
// Host only, integer arithmetic, deterministic tie-breaks.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <functional>
#include <queue>
#include <utility>
#include <vector>

#include "errors.h"
#include "libra.h"

using libra::fail;

extern "C" int libra_vrsp(const int64_t *lengths, int64_t num_samples, const int64_t *seq_cu,
                          int64_t num_seqs, int32_t pool_size, int64_t *order,
                          int64_t *pool_load, int64_t *seq_work) {
  libra::last_error_text().clear();
  if (num_seqs < 1 || pool_size < 1 || num_seqs % pool_size)
    return fail(LIBRA_EINVAL, "pool size %d must divide the window of %lld sequences",
                pool_size, (long long)num_seqs);
  if (num_samples < 0 || (num_samples > 0 && !lengths) || !seq_cu || !order)
    return fail(LIBRA_EINVAL, "NULL argument");
  if (seq_cu[0] != 0 || seq_cu[num_seqs] != num_samples)
    return fail(LIBRA_EINVAL, "seq_cu must run from 0 to num_samples");
  // Eq. 4: F_i = sum_j l_ij^2
  std::vector<int64_t> F((size_t)num_seqs);
  for (int64_t i = 0; i < num_seqs; ++i) {
    if (seq_cu[i + 1] < seq_cu[i])
      return fail(LIBRA_EINVAL, "seq_cu decreases at sequence %lld", (long long)i);
    __int128 f = 0;
    for (int64_t j = seq_cu[i]; j < seq_cu[i + 1]; ++j) {
      if (lengths[j] < 1) return fail(LIBRA_EINVAL, "sample %lld has length < 1", (long long)j);
      f += (__int128)lengths[j] * lengths[j];
      if (f > INT64_MAX) return fail(LIBRA_EOVERFLOW, "workload of sequence %lld", (long long)i);
    }
    F[(size_t)i] = (int64_t)f;
  }
  // decreasing F, then increasing index
  std::vector<int64_t> by_weight((size_t)num_seqs);
  for (int64_t i = 0; i < num_seqs; ++i) by_weight[(size_t)i] = i;
  std::sort(by_weight.begin(), by_weight.end(), [&](int64_t a, int64_t b) {
    return F[(size_t)a] != F[(size_t)b] ? F[(size_t)a] > F[(size_t)b] : a < b;
  });
  // min-heap of (load, pool) over the pools that are not full
  const int64_t K = num_seqs / pool_size;
  using Entry = std::pair<int64_t, int64_t>;
  std::priority_queue<Entry, std::vector<Entry>, std::greater<Entry>> heap;
  for (int64_t k = 0; k < K; ++k) heap.push({0, k});
  std::vector<int64_t> load((size_t)K, 0), filled((size_t)K, 0);
  for (int64_t i : by_weight) {
    const Entry top = heap.top();
    heap.pop();
    const int64_t k = top.second;
    if (load[(size_t)k] > INT64_MAX - F[(size_t)i])
      return fail(LIBRA_EOVERFLOW, "load of pool %lld", (long long)k);
    load[(size_t)k] += F[(size_t)i];
    // pools are concatenated in index order: pool k owns output slots
    // [k P, (k + 1) P), filled in placement order
    order[k * pool_size + filled[(size_t)k]] = i;
    if (++filled[(size_t)k] < pool_size) heap.push({load[(size_t)k], k});
  }
  if (pool_load) std::memcpy(pool_load, load.data(), sizeof(int64_t) * (size_t)K);
  if (seq_work) std::memcpy(seq_work, F.data(), sizeof(int64_t) * (size_t)num_seqs);
  return LIBRA_OK;
}
