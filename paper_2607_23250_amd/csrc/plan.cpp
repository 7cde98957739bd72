// Host planner: SH-Tiles (Eq. 5), tile cost (Eq. 6), KV groups (Eq. 7),
// communication increment (Eq. 8) and the communication-aware placement of
// Algorithm 2 (Sec. 4.3 of the Libra paper).  Pure integer arithmetic; the
// capacity test of Algorithm 2 is evaluated exactly with 128-bit products.
#include <algorithm>
#include <cstdint>
#include <cstring>
#include <numeric>
#include <vector>

#include "errors.h"
#include "libra.h"

namespace libra {

std::string &last_error_text() {
  static thread_local std::string s;
  return s;
}

namespace {

using i64 = int64_t;
using i128 = __int128;

struct Tile {
  i64 q_begin, q_end, q_row, cost;
  int32_t pack, home, id, shard;
  i64 s_first, s_last;   // K(t): samples s_first..s_last intersect the block
  i64 vq;                // V_Q(t) = V_O(t) bytes
};

// Rank holding chunk c of a pack under the head+tail CP layout.
inline int32_t zigzag_rank(i64 c, int32_t cp) {
  return static_cast<int32_t>(c < cp ? c : 2 * cp - 1 - c);
}

bool fits_i64(i128 x) { return x >= INT64_MIN && x <= INT64_MAX; }

int validate(const libra_plan_cfg_t *cfg, const int64_t *lengths, int64_t n,
             const int64_t *cu, const int64_t *pack_cu) {
  if (!cfg) return fail(LIBRA_EINVAL, "cfg is NULL");
  const auto &c = *cfg;
  if (c.block_tokens < 1 || c.head_shards < 1 || c.num_packs < 1 || c.cp < 1 ||
      c.num_q_heads < 1 || c.num_kv_heads < 1 || c.head_dim < 1 || c.elem_bytes < 1 ||
      c.tau_den < 1 || c.tau_num < 0)
    return fail(LIBRA_EINVAL, "cfg fields must be positive (tau_num >= 0)");
  if (c.num_q_heads % c.num_kv_heads)
    return fail(LIBRA_EINVAL, "num_kv_heads (%d) must divide num_q_heads (%d)", c.num_kv_heads,
                c.num_q_heads);
  if (c.num_q_heads % c.head_shards)
    return fail(LIBRA_EINVAL, "head_shards (%d) must divide num_q_heads (%d)", c.head_shards,
                c.num_q_heads);
  if (c.num_kv_heads % c.head_shards && c.head_shards % c.num_kv_heads)
    return fail(LIBRA_EINVAL, "head_shards (%d) and num_kv_heads (%d) must divide one another",
                c.head_shards, c.num_kv_heads);
  if ((i64)c.num_packs * c.cp > INT32_MAX) return fail(LIBRA_EINVAL, "too many workers");
  if (n < 1 || !lengths || !cu || !pack_cu)
    return fail(LIBRA_EINVAL, "need num_samples >= 1 and non-NULL lengths/cu_seqlens/pack_cu");
  if (cu[0] != 0) return fail(LIBRA_EINVAL, "cu_seqlens[0] must be 0");
  for (i64 j = 0; j < n; ++j) {
    if (lengths[j] < 1) return fail(LIBRA_EINVAL, "lengths[%lld] < 1", (long long)j);
    if (cu[j + 1] - cu[j] != lengths[j])
      return fail(LIBRA_EINVAL, "cu_seqlens[%lld] does not match lengths", (long long)(j + 1));
  }
  if (pack_cu[0] != 0 || pack_cu[c.num_packs] != cu[n])
    return fail(LIBRA_EINVAL, "pack_cu must start at 0 and end at cu_seqlens[n]");
  i64 j = 0;
  for (int32_t p = 0; p < c.num_packs; ++p) {
    const i64 len = pack_cu[p + 1] - pack_cu[p];
    if (len < 1) return fail(LIBRA_EINVAL, "pack %d is empty", p);
    if (len % (2 * (i64)c.cp))
      return fail(LIBRA_EINVAL, "pack %d length %lld is not a multiple of 2*cp", p,
                  (long long)len);
    while (j < n && cu[j] < pack_cu[p + 1]) ++j;
    if (cu[j] != pack_cu[p + 1])
      return fail(LIBRA_EINVAL, "pack boundary %lld is not a sample boundary",
                  (long long)pack_cu[p + 1]);
  }
  return LIBRA_OK;
}

}  // namespace
}  // namespace libra

using namespace libra;

extern "C" const char *libra_strerror(int code) {
  switch (code) {
    case LIBRA_OK: return "ok";
    case LIBRA_EINVAL: return "invalid argument";
    case LIBRA_ENOSPC: return "buffer too small";
    case LIBRA_EUNSUPPORTED: return "unsupported configuration";
    case LIBRA_EOVERFLOW: return "integer overflow";
    case LIBRA_EHIP: return "HIP runtime error";
    default: return "unknown error";
  }
}

extern "C" const char *libra_last_error(void) { return last_error_text().c_str(); }

extern "C" int libra_plan(const libra_plan_cfg_t *cfg, const int64_t *lengths,
                          int64_t num_samples, const int64_t *cu, const int64_t *pack_cu,
                          const int64_t *q_ranges, int32_t num_q_ranges, libra_tile_t *out,
                          int64_t tiles_cap, int64_t *num_tiles, int64_t *worker_load,
                          int64_t *worker_bytes) {
  last_error_text().clear();
  if (int rc = validate(cfg, lengths, num_samples, cu, pack_cu)) return rc;
  if (!num_tiles) return fail(LIBRA_EINVAL, "num_tiles is NULL");
  if (num_q_ranges < 0 || (num_q_ranges > 0 && !q_ranges))
    return fail(LIBRA_EINVAL, "q_ranges is NULL or num_q_ranges < 0");
  const auto &c = *cfg;
  const i64 n = num_samples, B = c.block_tokens, H = c.head_shards, CP = c.cp;
  const i64 V = (i64)c.num_packs * CP;
  const i64 heads = c.num_q_heads / H;
  const i64 kvh = std::max<i64>(1, c.num_kv_heads / H);
  const i64 total = cu[n];
  for (int32_t r = 0; r < num_q_ranges; ++r) {
    const i64 b = q_ranges[2 * r], e = q_ranges[2 * r + 1];
    if (b < 0 || e > total || b >= e || (r > 0 && b < q_ranges[2 * r - 1]))
      return fail(LIBRA_EINVAL, "q_ranges must be sorted, disjoint, non-empty and in range");
  }

  // Eq. 5 / Eq. 6 / Eq. 7: walk the blocks of every pack in position order.
  std::vector<Tile> tiles;
  i64 gb = 0, q_row = 0, j = 0, rr = 0;
  for (int32_t p = 0; p < c.num_packs; ++p) {
    const i64 off = pack_cu[p], end = pack_cu[p + 1], chunk = (end - off) / (2 * CP);
    for (i64 lo = off; lo < end; lo += B, ++gb) {
      const i64 hi = std::min(end, lo + B);
      if (num_q_ranges > 0) {
        while (rr < num_q_ranges && q_ranges[2 * rr + 1] <= lo) ++rr;
        const bool inside = rr < num_q_ranges && q_ranges[2 * rr] <= lo && hi <= q_ranges[2 * rr + 1];
        const bool touches = rr < num_q_ranges && q_ranges[2 * rr] < hi;
        if (touches && !inside)
          return fail(LIBRA_EINVAL, "q_ranges cut block [%lld, %lld); ranges must hold whole blocks",
                      (long long)lo, (long long)hi);
        if (!inside) continue;
      }
      while (cu[j + 1] <= lo) ++j;       // first sample intersecting [lo, hi)
      i128 pairs = 0;
      i64 jj = j;
      for (; jj < n && cu[jj] < hi; ++jj) {
        const i64 a = std::max(lo, cu[jj]) - cu[jj];
        const i64 e = std::min(hi, cu[jj + 1]) - cu[jj];
        pairs += (i128)e * (e + 1) / 2 - (i128)a * (a + 1) / 2;
      }
      const i128 cost = pairs * heads;
      const i128 vq = (i128)(hi - lo) * heads * c.head_dim * c.elem_bytes;
      if (!fits_i64(cost) || !fits_i64(2 * vq))
        return fail(LIBRA_EOVERFLOW, "tile cost or byte size overflows int64");
      const int32_t home = (int32_t)(p * CP + zigzag_rank((lo - off) / chunk, (int32_t)CP));
      for (i64 h = 0; h < H; ++h) {
        const i128 id = (i128)gb * H + h;
        if (id > INT32_MAX) return fail(LIBRA_EOVERFLOW, "tile id overflows int32");
        tiles.push_back(Tile{lo, hi, q_row, (i64)cost, p, home, (int32_t)id, (int32_t)h, j,
                             jj - 1, (i64)vq});
      }
      q_row += hi - lo;
    }
  }
  if (num_q_ranges > 0) {
    // every range must be covered by whole blocks
    i64 covered = 0, want = 0;
    for (int32_t r = 0; r < num_q_ranges; ++r) want += q_ranges[2 * r + 1] - q_ranges[2 * r];
    for (const Tile &t : tiles)
      if (t.shard == 0) covered += t.q_end - t.q_begin;
    if (covered != want)
      return fail(LIBRA_EINVAL, "q_ranges must consist of whole blocks");
  }
  const i64 T = (i64)tiles.size();
  *num_tiles = T;
  if (!out && !worker_load) return LIBRA_OK;
  if (out && tiles_cap < T)
    return fail(LIBRA_ENOSPC, "tiles_cap %lld < %lld tiles", (long long)tiles_cap, (long long)T);

  // KV group bytes V_g and the initial resident sets C_r.
  std::vector<i64> vg(n);
  for (i64 s = 0; s < n; ++s) {
    const i128 b = (i128)lengths[s] * kvh * c.head_dim * c.elem_bytes * 2;
    if (!fits_i64(b)) return fail(LIBRA_EOVERFLOW, "KV group bytes overflow int64");
    vg[s] = (i64)b;
  }
  // resident[(s * H + h) * V + r]
  std::vector<uint8_t> resident((size_t)(n * H * V), 0);
  {
    i64 p = 0;
    for (i64 s = 0; s < n; ++s) {
      while (pack_cu[p + 1] <= cu[s]) ++p;
      const i64 off = pack_cu[p], chunk = (pack_cu[p + 1] - off) / (2 * CP);
      const i64 c0 = (cu[s] - off) / chunk, c1 = (cu[s + 1] - 1 - off) / chunk;
      const int32_t r0 = zigzag_rank(c0, (int32_t)CP);
      bool whole = true;
      for (i64 cc = c0 + 1; cc <= c1 && whole; ++cc) whole = zigzag_rank(cc, (int32_t)CP) == r0;
      if (whole)
        for (i64 h = 0; h < H; ++h) resident[(size_t)((s * H + h) * V + p * CP + r0)] = 1;
    }
  }

  // Algorithm 2.
  i128 S = 0;
  for (const Tile &t : tiles) S += t.cost;
  const i128 cap_rhs = (i128)(c.tau_den + c.tau_num) * S;   // (1+tau)*S*tau_den
  const i128 cap_lhs_mul = (i128)c.tau_den * V;
  std::vector<i64> order(T);
  std::iota(order.begin(), order.end(), 0);
  std::sort(order.begin(), order.end(), [&](i64 a, i64 b) {
    if (tiles[a].cost != tiles[b].cost) return tiles[a].cost > tiles[b].cost;
    return tiles[a].id < tiles[b].id;
  });
  std::vector<i64> load(V, 0), received(V, 0);
  std::vector<int32_t> assign(T, -1);
  std::vector<i64> delta(V);
  for (i64 idx : order) {
    const Tile &t = tiles[idx];
    bool any_feasible = false;
    for (i64 r = 0; r < V; ++r) {
      i128 d = (r == t.home) ? 0 : 2 * (i128)t.vq;
      for (i64 s = t.s_first; s <= t.s_last; ++s)
        if (!resident[(size_t)((s * H + t.shard) * V + r)]) d += vg[s];
      if (!fits_i64(d)) return fail(LIBRA_EOVERFLOW, "communication bytes overflow int64");
      delta[r] = (i64)d;
      any_feasible |= cap_lhs_mul * ((i128)load[r] + t.cost) <= cap_rhs;
    }
    i64 best = -1;
    for (i64 r = 0; r < V; ++r) {
      if (any_feasible) {
        if (cap_lhs_mul * ((i128)load[r] + t.cost) > cap_rhs) continue;
        if (best < 0 || delta[r] < delta[best] ||
            (delta[r] == delta[best] && load[r] < load[best]))
          best = r;
      } else {
        if (best < 0 || load[r] < load[best] ||
            (load[r] == load[best] && delta[r] < delta[best]))
          best = r;
      }
    }
    assign[idx] = (int32_t)best;
    if (!fits_i64((i128)load[best] + t.cost)) return fail(LIBRA_EOVERFLOW, "load overflows");
    if (!fits_i64((i128)received[best] + delta[best]))
      return fail(LIBRA_EOVERFLOW, "received bytes overflow int64");
    load[best] += t.cost;
    received[best] += delta[best];
    for (i64 s = t.s_first; s <= t.s_last; ++s)
      resident[(size_t)((s * H + t.shard) * V + best)] = 1;
  }

  if (out) {
    for (i64 i = 0; i < T; ++i) {
      const Tile &t = tiles[i];
      libra_tile_t &o = out[i];
      o.q_begin = t.q_begin;
      o.q_end = t.q_end;
      o.q_row = t.q_row;
      o.cost = t.cost;
      o.head_begin = (int32_t)(t.shard * heads);
      o.head_end = (int32_t)((t.shard + 1) * heads);
      o.pack = t.pack;
      o.home = t.home;
      o.worker = assign[i];
      o.id = t.id;
    }
  }
  if (worker_load) std::memcpy(worker_load, load.data(), sizeof(i64) * V);
  if (worker_bytes) std::memcpy(worker_bytes, received.data(), sizeof(i64) * V);
  return LIBRA_OK;
}
