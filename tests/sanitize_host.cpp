// Host-code check under AddressSanitizer and UndefinedBehaviorSanitizer: the
// planner (libra_plan) and VRSP (libra_vrsp) on random valid inputs, size
// queries, undersized outputs and malformed arguments.  Built and run by
// tests/test_host_sanitizers.py with g++ (no GPU code is involved); any
// sanitizer report aborts with a non-zero exit.
#include <algorithm>
#include <cstdint>
#include <cstdlib>
#include <cstdio>
#include <vector>

#include "libra.h"

namespace {

uint64_t rng_state = 0x9E3779B97F4A7C15ull;
uint64_t next_u64() {   // xorshift64*
  rng_state ^= rng_state >> 12;
  rng_state ^= rng_state << 25;
  rng_state ^= rng_state >> 27;
  return rng_state * 0x2545F4914F6CDD1Dull;
}
int64_t rnd(int64_t lo, int64_t hi) { return lo + (int64_t)(next_u64() % (uint64_t)(hi - lo + 1)); }

int fails = 0;
void expect(bool ok, const char *what, int iter) {
  if (!ok) {
    std::fprintf(stderr, "case %d: %s\n", iter, what);
    ++fails;
  }
}

void plan_case(int it) {
  const int32_t layouts[][3] = {{2, 1, 2}, {4, 1, 2}, {8, 2, 2}, {8, 2, 4}, {32, 4, 2},
                                {12, 4, 4}, {4, 4, 1}, {32, 2, 8}, {6, 3, 3}, {64, 4, 16}};
  const auto &lay = layouts[rnd(0, 9)];
  libra_plan_cfg_t cfg{};
  cfg.num_q_heads = lay[0];
  cfg.num_kv_heads = lay[1];
  cfg.head_shards = lay[2];
  cfg.cp = (int32_t)rnd(1, 4);
  cfg.num_packs = (int32_t)rnd(1, 4);
  cfg.block_tokens = (int32_t)rnd(1, 300);
  cfg.head_dim = (int32_t)(rnd(0, 1) ? 64 : 128);
  cfg.elem_bytes = 2;
  cfg.tau_num = (int32_t)rnd(0, 10);
  cfg.tau_den = (int32_t)rnd(1, 100);
  std::vector<int64_t> lengths, cu{0}, pack_cu{0};
  for (int p = 0; p < cfg.num_packs; ++p) {
    int64_t room = 2 * cfg.cp * rnd(1, 120);
    while (room > 0) {
      const int64_t n = std::min<int64_t>(room, rnd(0, 4) ? rnd(1, 400) : rnd(1, 8));
      lengths.push_back(n);
      cu.push_back(cu.back() + n);
      room -= n;
    }
    pack_cu.push_back(cu.back());
  }
  const int64_t n = (int64_t)lengths.size();
  // whole-block query ranges on half of the cases
  std::vector<int64_t> qr;
  if (rnd(0, 1)) {
    for (int p = 0; p < cfg.num_packs; ++p)
      for (int64_t lo = pack_cu[p]; lo < pack_cu[p + 1]; lo += cfg.block_tokens) {
        const int64_t hi = std::min(pack_cu[p + 1], lo + cfg.block_tokens);
        if (rnd(0, 1)) continue;
        if (!qr.empty() && qr.back() == lo) qr.back() = hi;
        else { qr.push_back(lo); qr.push_back(hi); }
      }
  }
  const int32_t R = (int32_t)(qr.size() / 2);
  int64_t T = -1;
  int rc = libra_plan(&cfg, lengths.data(), n, cu.data(), pack_cu.data(), R ? qr.data() : nullptr,
                      R, nullptr, 0, &T, nullptr, nullptr);
  expect(rc == LIBRA_OK && T >= 0, "size query", it);
  const int64_t V = (int64_t)cfg.num_packs * cfg.cp;
  std::vector<libra_tile_t> tiles((size_t)T + 1);
  std::vector<int64_t> load((size_t)V), bytes((size_t)V);
  if (T > 0) {
    int64_t T2 = -1;
    rc = libra_plan(&cfg, lengths.data(), n, cu.data(), pack_cu.data(), R ? qr.data() : nullptr,
                    R, tiles.data(), T - 1, &T2, load.data(), bytes.data());
    expect(rc == LIBRA_ENOSPC && T2 == T, "undersized tile buffer", it);
  }
  rc = libra_plan(&cfg, lengths.data(), n, cu.data(), pack_cu.data(), R ? qr.data() : nullptr, R,
                  tiles.data(), T, &T, load.data(), bytes.data());
  expect(rc == LIBRA_OK, "plan", it);
  int64_t sum = 0, lsum = 0;
  for (int64_t t = 0; t < T; ++t) {
    sum += tiles[(size_t)t].cost;
    expect(tiles[(size_t)t].worker >= 0 && tiles[(size_t)t].worker < V, "worker range", it);
  }
  for (int64_t r = 0; r < V; ++r) lsum += load[(size_t)r];
  expect(sum == lsum, "loads sum to the costs", it);
  // malformed inputs
  libra_plan_cfg_t bad = cfg;
  bad.head_shards = cfg.num_q_heads + 1;
  expect(libra_plan(&bad, lengths.data(), n, cu.data(), pack_cu.data(), nullptr, 0, nullptr, 0,
                    &T, nullptr, nullptr) == LIBRA_EINVAL, "bad head shards", it);
  std::vector<int64_t> bad_cu = cu;
  bad_cu[(size_t)n] += 1;
  expect(libra_plan(&cfg, lengths.data(), n, bad_cu.data(), pack_cu.data(), nullptr, 0, nullptr, 0,
                    &T, nullptr, nullptr) == LIBRA_EINVAL, "inconsistent cu_seqlens", it);
  expect(libra_plan(nullptr, lengths.data(), n, cu.data(), pack_cu.data(), nullptr, 0, nullptr, 0,
                    &T, nullptr, nullptr) == LIBRA_EINVAL, "NULL cfg", it);
  if (n > 0 && cfg.block_tokens > 1) {
    const int64_t cut[2] = {0, 1};   // a range that cuts the first block
    expect(libra_plan(&cfg, lengths.data(), n, cu.data(), pack_cu.data(), cut, 1, nullptr, 0, &T,
                      nullptr, nullptr) == LIBRA_EINVAL, "range cutting a block", it);
  }
}

void vrsp_case(int it) {
  const int32_t P = (int32_t)rnd(1, 8);
  const int64_t S = P * rnd(1, 8);
  std::vector<int64_t> lengths, seq_cu{0};
  for (int64_t s = 0; s < S; ++s) {
    const int64_t k = rnd(0, 6);
    for (int64_t i = 0; i < k; ++i) lengths.push_back(rnd(1, 5000));
    seq_cu.push_back((int64_t)lengths.size());
  }
  std::vector<int64_t> order((size_t)S), pool((size_t)(S / P)), work((size_t)S);
  const int64_t ns = (int64_t)lengths.size();
  int rc = libra_vrsp(ns ? lengths.data() : nullptr, ns, seq_cu.data(), S, P, order.data(),
                      pool.data(), work.data());
  if (ns == 0) return;   // no samples: the call may reject the empty window
  expect(rc == LIBRA_OK, "vrsp", it);
  std::vector<int> seen((size_t)S, 0);
  for (int64_t i = 0; i < S; ++i)
    if (order[(size_t)i] >= 0 && order[(size_t)i] < S) ++seen[(size_t)order[(size_t)i]];
  for (int64_t i = 0; i < S; ++i) expect(seen[(size_t)i] == 1, "vrsp permutation", it);
  expect(libra_vrsp(lengths.data(), ns, seq_cu.data(), S, P + (S % (P + 1) ? 1 : 0) + S,
                    order.data(), nullptr, nullptr) == LIBRA_EINVAL, "pool size not dividing",
         it);
}

}  // namespace

int main(int argc, char **argv) {
  const int iters = argc > 1 ? std::atoi(argv[1]) : 500;
  for (int it = 0; it < iters; ++it) {
    plan_case(it);
    vrsp_case(it);
  }
  std::printf("%d cases, %d failures\n", iters, fails);
  return fails ? 1 : 0;
}
