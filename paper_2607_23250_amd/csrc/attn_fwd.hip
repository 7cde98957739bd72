// Forward pass of document-masked causal attention over SH-Tiles (gfx950).
//
// What is computed: Eq. 1 of the paper under the block-diagonal causal mask of
// packing (Sec. 2.3), for the (row, query head) pairs covered by a list of
// SH-Tiles (Sec. 4.3.1).  Each tile is cut into work items on the device; a
// persistent kernel walks the items longest-first.
//
// Kernel structure (one work item = up to 4 query heads of one KV group x 32
// rows per head, or fewer heads x more rows; 4 waves, one (head, 32 rows) each):
//   * K and V blocks of 64 keys are staged in LDS as rows, double-buffered;
//     blocks are anchored at the sample start and only the row's own sample
//     is visited, so cross-document blocks are never touched.
//   * S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (keys on M, queries on N), so
//     that every lane owns one query: the row max / row sum of the online
//     softmax are 32 in-lane values plus one exchange with lane ^ 32.
//   * O^T += V^T P^T with the same instruction; P^T comes straight from the
//     S^T accumulators (bf16), V^T from the row-major V tile through the LDS
//     transpose reads.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "attn_common.h"
#include "errors.h"

namespace libra {

// ---------------------------------------------------------------------------
// Work items: every tile is split into sample fragments; every fragment into
// items of (<= 4 heads of one KV group) x (32 * 4 / heads rows), starting at
// the fragment's first row.  The enumeration goes by 32-row windows of a tile:
// f(item, key blocks) is called for the items whose first row lies in rows
// [wa, wb) of tile t (wb - wa <= 32, so at most one item per fragment and
// head chunk), which spreads a tile's items over many threads.
template <typename F>
__device__ void for_each_fwd_item_in(const libra_tile_t &t, int64_t wa, int64_t wb,
                                     const int64_t *cu, int64_t n, int G, F &&f) {
  int64_t j = upper_bound64(cu, n, wa) - 1;
  for (; j < n && cu[j] < wb; ++j) {
    const int64_t pb = t.q_begin > cu[j] ? t.q_begin : cu[j];
    const int64_t pe = t.q_end < cu[j + 1] ? t.q_end : cu[j + 1];
    const int32_t row0 = (int32_t)(t.q_row + (pb - t.q_begin));
    const int32_t qloc0 = (int32_t)(pb - cu[j]);
    const int32_t nfrag = (int32_t)(pe - pb);
    const int64_t lim = wb < pe ? wb : pe;
    for (int g = t.head_begin / G; g * G < t.head_end; ++g) {
      const int hl = max(t.head_begin, g * G), hh = min(t.head_end, (g + 1) * G);
      for (int h0 = hl; h0 < hh; h0 += 4) {
        const int nh = min(4, hh - h0);
        const int rows_per = kRows * (4 / nh);
        // first item start pb + k rows_per at or after wa
        int64_t k = wa > pb ? (wa - pb + rows_per - 1) / rows_per : 0;
        for (; pb + k * rows_per < lim; ++k) {
          const int32_t rb = (int32_t)(k * rows_per);
          const int nrows = min(rows_per, nfrag - rb);
          const int32_t nkb = (qloc0 + rb + nrows - 1) / kFwdBN + 1;
          FwdItem it{row0 + rb, qloc0 + rb, (int32_t)j, h0, nh, nrows, g, 0, nkb, -1, 0, 0};
          f(it, nkb);
        }
      }
    }
  }
}

// One workgroup: every tile's items, longest-first, one queue per XCD keyed
// by (KV head, head chunk) so that an XCD streams few K/V sequences.  Tiles
// outside the buffers are skipped, and counted in hdr[kBadTiles] when
// `count_bad` is set (the backward counts them in its own preparation pass).
//
// Split K: when there are fewer than two items per workgroup of the `grid`
// that runs them (few rows and heads against long samples), and with
// `idle_only` only when whole rounds of `grid` items would leave more than a
// tenth of the workgroups idle, the key blocks that all rows of an item
// attend in full (below its first row's block kd) are cut into ranges of C
// blocks, about four items per workgroup in all;
// the last range also takes the blocks from kd on, so that every row has a
// key in the first block of every range.  Items with kd < 2 C stay whole.
// Each part writes a partial result to its own slot (max_parts slots;
// max_parts = 0 never splits) and fwd_combine_kernel merges the parts of
// every split item.  C is at least kFwdSplitMinBlocks and doubles until the
// parts fit the slots.
__global__ __launch_bounds__(kPrepThreads) void prep_fwd_kernel(
    const int64_t *__restrict__ cu, int64_t n, const libra_tile_t *__restrict__ tiles, int64_t T,
    int h_q, int h_kv, int64_t n_q, int64_t n_kv, int32_t *__restrict__ hdr,
    FwdItem *__restrict__ items, int64_t max_items, int count_bad, int grid, int max_parts,
    int idle_only, FwdSplit *__restrict__ splits) {
  __shared__ int32_t hist[kXcds * kQBuckets];
  __shared__ int32_t part[kPrepThreads];
  __shared__ unsigned long long s_wmax, s_items, s_work, s_parts, s_pairs;
  __shared__ int32_t s_chunk, s_nslot, s_nsplit;
  const int tid = threadIdx.x;
  const int G = h_q / h_kv;
  const int chunks = (G + 3) / 4;                    // head chunks per KV group
  const int keys = h_kv * chunks;
  const int R = keys >= kXcds ? 1 : kXcds / keys;    // queues per key
  if (tid == 0) {
    if (count_bad) hdr[kBadTiles] = 0;
    hdr[kFwdSplits] = 0;
    hdr[kFwdSplits + 1] = 0;
    s_wmax = 0;
    s_pairs = 0;
    s_items = 0;
    s_work = 0;
    s_chunk = 0;
    s_nslot = 0;
    s_nsplit = 0;
  }
  __threadfence();
  __syncthreads();
  // bad tiles, and the 32-row windows of the longest good tile
  int bad = 0;
  unsigned long long wm = 0, pairs = 0;
  for (int64_t t = tid; t < T; t += kPrepThreads) {
    const libra_tile_t tl = tiles[t];
    if (!tile_ok(tl, n_q, n_kv, h_q)) {
      ++bad;
      continue;
    }
    const unsigned long long w = (unsigned long long)((tl.q_end - tl.q_begin + kRows - 1) / kRows);
    wm = w > wm ? w : wm;
    pairs += (unsigned long long)(tl.q_end - tl.q_begin) * (unsigned long long)(tl.head_end - tl.head_begin);
  }
  if (bad && count_bad) atomicAdd(&hdr[kBadTiles], bad);
  if (wm) atomicMax(&s_wmax, wm);
  if (pairs) atomicAdd(&s_pairs, pairs);
  __syncthreads();
  const int64_t wmax = (int64_t)s_wmax;
  // every whole item once: f(item, queue)
  auto whole = [&](auto &&f) {
    for (int64_t v = tid; v < T * wmax; v += kPrepThreads) {
      const int64_t t = v / wmax, w = v % wmax;
      const libra_tile_t tl = tiles[t];
      if (!tile_ok(tl, n_q, n_kv, h_q)) continue;
      const int64_t wa = tl.q_begin + (int64_t)kRows * w;
      if (wa >= tl.q_end) continue;
      const int64_t wb = wa + kRows < tl.q_end ? wa + kRows : tl.q_end;
      for_each_fwd_item_in(tl, wa, wb, cu, n, G, [&](const FwdItem &it, int) {
        const int key = it.g * chunks + (it.head0 - it.g * G) / 4;
        f(it, (key * R + (it.q_row0 / 128) % R) % kXcds);
      });
    }
  };
  // an item covers at most 128 (row, head) pairs: with pairs / 128 items or
  // more there are enough for the grid, and the item count is not needed
  if (max_parts > 0 && s_pairs / 128 < 2ull * (unsigned long long)grid) {
    whole([&](const FwdItem &it, int) {
      atomicAdd(&s_items, 1ull);
      atomicAdd(&s_work, (unsigned long long)it.kb1);
    });
    __syncthreads();
    const unsigned long long n_items = s_items, work = s_work, gr = (unsigned long long)grid;
    // rounds of `grid` items fill less than 90% of the workgroups
    const bool idle = n_items * 10 < (n_items + gr - 1) / gr * gr * 9;
    if (n_items > 0 && n_items < 2 * gr && (idle || !idle_only)) {
      long long c = (long long)((work + 4ull * grid - 1) / (4ull * grid));
      c = c > kFwdSplitMinBlocks ? c : kFwdSplitMinBlocks;
      for (; c < (1ll << 30); c *= 2) {   // at most ~30 rounds; the first fits by construction
        if (tid == 0) s_parts = 0;
        __syncthreads();
        whole([&](const FwdItem &it, int) {
          const long long np = (it.q_loc0 / kFwdBN) / c;
          if (np >= 2) atomicAdd(&s_parts, (unsigned long long)np);
        });
        __syncthreads();
        const bool fits = s_parts <= (unsigned long long)max_parts;
        __syncthreads();
        if (fits) break;
      }
      if (tid == 0) s_chunk = (int32_t)(c < (1ll << 30) ? c : 0);
    }
    __syncthreads();
  }
  const int chunk = s_chunk;   // 0: no item is split
  auto each = [&](auto &&f, bool scatter) {
    whole([&](const FwdItem &it, int x) {
      const int np = chunk ? (it.q_loc0 / kFwdBN) / chunk : 0;
      if (np < 2) {
        f(it, (int64_t)it.kb1, x);
        return;
      }
      int32_t base = 0;
      if (scatter) {
        base = atomicAdd(&s_nslot, np);
        splits[atomicAdd(&s_nsplit, 1)] = FwdSplit{it, base, np, 0, 0};
      }
      for (int p = 0; p < np; ++p) {
        FwdItem ip = it;
        ip.kb0 = p * chunk;
        ip.kb1 = p + 1 < np ? (p + 1) * chunk : it.kb1;
        ip.slot = base + p;
        f(ip, (int64_t)(ip.kb1 - ip.kb0), x);
      }
    });
  };
  build_queues<FwdItem>(each, hist, part, hdr, kFwdQ, items, max_items);
  __syncthreads();
  if (tid == 0) {
    hdr[kFwdSplits] = s_nsplit;
    hdr[kFwdSplits + 1] = s_nslot;
  }
}

// Merges the parts of every split item (hdr[kFwdSplits] records): per row,
// m = max_p m_p, l = sum_p l_p 2^(m_p - m), O = sum_p O_p 2^(m_p - m) / l and
// LSE = (m + log2 l) ln 2, the online-softmax recurrence applied across the
// key ranges.  Two threads per row (half of the head dimension each).
template <int D>
__global__ __launch_bounds__(256) void fwd_combine_kernel(
    const FwdSplit *__restrict__ splits, const int32_t *__restrict__ hdr,
    const float *__restrict__ parts, int h_q, int64_t n_q, bf16 *__restrict__ o,
    float *__restrict__ lse) {
  constexpr size_t PF = fwd_part_floats(D);
  const int count = hdr[kFwdSplits];
  const int tid = threadIdx.x, pr = tid >> 1, half = tid & 1;
  const int w = pr >> 5, r = pr & 31;   // wave slice and row of the item
  for (int e = blockIdx.x; e < count; e += gridDim.x) {
    const FwdSplit sp = splits[e];
    const FwdItem &it = sp.item;
    const int wrow0 = (w / it.nh) * kRows;
    const int wrows = min(max(it.nrows - wrow0, 0), kRows);
    if (r >= wrows) continue;
    const int head = it.head0 + (w % it.nh);
    const int64_t row = (int64_t)it.q_row0 + wrow0 + r;
    float m = -INFINITY;
    for (int p = 0; p < sp.parts; ++p) {
      const float *rec = parts + (size_t)(sp.base + p) * PF + (size_t)kFwdPartRows * D;
      m = fmaxf(m, rec[pr]);
    }
    float l = 0.f;
    float acc[D / 2];
#pragma unroll
    for (int i = 0; i < D / 2; ++i) acc[i] = 0.f;
    for (int p = 0; p < sp.parts; ++p) {
      const float *rec = parts + (size_t)(sp.base + p) * PF;
      const float mp = rec[(size_t)kFwdPartRows * D + pr];
      const float wgt = mp == -INFINITY ? 0.f : fast_exp2(mp - m);
      l += wgt * rec[(size_t)kFwdPartRows * D + kFwdPartRows + pr];
      const float4 *src = reinterpret_cast<const float4 *>(rec + (size_t)pr * D + half * (D / 2));
#pragma unroll
      for (int i = 0; i < D / 8; ++i) {
        const float4 x = src[i];
        acc[4 * i] += wgt * x.x;
        acc[4 * i + 1] += wgt * x.y;
        acc[4 * i + 2] += wgt * x.z;
        acc[4 * i + 3] += wgt * x.w;
      }
    }
    const float inv = 1.f / l;
    bf16 *op = o + ((size_t)row * h_q + head) * D + half * (D / 2);
#pragma unroll
    for (int i = 0; i < D / 16; ++i) {
      bf16x8 ov;
#pragma unroll
      for (int j = 0; j < 8; ++j) ov[j] = static_cast<bf16>(acc[8 * i + j] * inv);
      *reinterpret_cast<bf16x8 *>(op + 8 * i) = ov;
    }
    if (half == 0) lse[(size_t)head * n_q + row] = (m + __builtin_amdgcn_logf(l)) * kLn2;
  }
}

// ---------------------------------------------------------------------------
template <int D>
struct FwdShape {
  static constexpr int KC = D / 8;            // 16-byte columns of a K / V row
  static constexpr int K_EL = kFwdBN * D;
  static constexpr int STAGE = 2 * K_EL;      // K and V rows of one key block
  static constexpr int NK = kFwdBN * KC / 64 / kWaves;   // wave loads of 1 KB per tile
  static constexpr size_t SMEM = 2 * STAGE * sizeof(bf16);
};

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ k, const bf16 *__restrict__ v,
    const int64_t *__restrict__ cu, const FwdItem *__restrict__ items, int32_t *__restrict__ hdr,
    int h_q, int h_kv, int64_t n_q, int64_t n_kv, float c2,
    bf16 *__restrict__ o, float *__restrict__ lse, float *__restrict__ parts) {
  using S = FwdShape<D>;
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  __shared__ int32_t s_item;
  const int tid = threadIdx.x, l = tid & 63, ln = l & 31, kg = l >> 5;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index (uniform)
  int q_serve = xcd_of_workgroup(), q_left = kXcds;
  // per-lane LDS offsets (elements) of the operand reads, fixed for the kernel
  // K rows perm32(ln) for S^T; transpose reads of the V tile for the V^T
  // operand of O^T (rows = keys, as in the dQ kernel's K^T)
  const int prow = perm32(ln);
  int koff[D / 16], troff[D / 32][2];
  static_for<D / 16>([&](auto c) { koff[c] = prow * D + 8 * swt<S::KC>(prow, 2 * c + kg); });
  {
    const int grp = l >> 4, i = (l & 15) >> 2, r = l & 3;
    static_for<D / 32>([&](auto dt) {
      static_for<2>([&](auto hf) {
        const int row = 8 * (grp >> 1) + 4 * hf + i;
        const int chunk = 4 * dt + 2 * (grp & 1) + (r & 1);
        troff[dt][hf] = row * D + 8 * swt<S::KC>(row, chunk) + 4 * (r >> 1);
      });
    });
  }
  // staging: wave load u covers rows (w + 4u) * 64 / KC + l / KC of a tile;
  // k_lane[u] is the lane's byte offset from the block's first K (V) row
  uint32_t k_lane[S::NK];
  static_for<S::NK>([&](auto u) {
    const int r = (w + kWaves * u) * (64 / S::KC) + l / S::KC;
    k_lane[u] = 2u * (uint32_t)(r * h_kv * D + 8 * swt<S::KC>(r, l % S::KC));
  });

  for (;;) {
    if (tid == 0) s_item = take_item(hdr, kFwdQ, q_serve, q_left);
    __syncthreads();
    const int idx = __builtin_amdgcn_readfirstlane(s_item);
    if (idx < 0) break;
    const FwdItem it = items[idx];
    const int64_t key0 = cu[it.sample];
    const int head = it.head0 + (w % it.nh);
    const int wrow0 = (w / it.nh) * kRows;
    const int wrows = min(max(it.nrows - wrow0, 0), kRows);
    const bool active = wrows > 0;
    const int my_r = active ? min(ln, wrows - 1) : 0;
    const int64_t row = (int64_t)it.q_row0 + wrow0 + my_r;
    const int qloc = it.q_loc0 + wrow0 + my_r;
    const int wave_qmin = it.q_loc0 + wrow0;
    const int kb0 = it.kb0, nkb = it.kb1;   // key blocks [kb0, nkb)
    const int wave_nkb = active ? (it.q_loc0 + wrow0 + wrows - 1) / kFwdBN + 1 : 0;

    bf16x8 qf[D / 16];
    if (active) {
      const bf16 *qp = q + ((size_t)row * h_q + head) * D + 8 * kg;
      static_for<D / 16>([&](auto c) { qf[c] = *reinterpret_cast<const bf16x8 *>(qp + 16 * c); });
    }
    f32x16 oacc[D / 32];
    static_for<D / 32>([&](auto dt) { static_for<16>([&](auto r) { oacc[dt][int(r)] = 0.f; }); });
    float m_run = -INFINITY, l_run = 0.f;

    // global -> LDS, asynchronous: the K (part 0) or V (part 1) rows of key
    // block b (keys past the buffer read the last key instead; keys past the
    // row are masked, and their V rows meet P = 0)
    auto issue = [&](int b, int buf, int part) {
      const bf16 *src = part ? v : k;
      bf16 *dst = smem + buf * S::STAGE + part * S::K_EL;
      const int64_t kbase = key0 + (int64_t)b * kFwdBN;
      if (kbase + kFwdBN <= n_kv) {
        // whole block inside the buffer: one SGPR base, fixed per-lane offsets;
        // wave load u lands 1 KiB x (w + kWaves u) into the tile
        const bf16 *base = src + ((size_t)kbase * h_kv + it.g) * D;
        const uint32_t ld = lds_addr(dst) + 1024u * w;
        static_for<S::NK / 4>([&](auto h) {
          constexpr uint32_t d = 4 * h * kWaves * 1024u, e = kWaves * 1024u;
          g2l16x4r(base, k_lane[4 * h], k_lane[4 * h + 1], k_lane[4 * h + 2], k_lane[4 * h + 3],
                   ld + d, ld + d + e, ld + d + 2 * e, ld + d + 3 * e);
        });
        static_for<S::NK % 4>([&](auto i) {
          constexpr int u = S::NK / 4 * 4 + i;
          g2l16s(base, k_lane[u], ld + u * kWaves * 1024u);
        });
        return;
      }
      // the last block of the buffer: keys past it read the last key (masked)
      static_for<S::NK>([&](auto u) {
        const int wl = w + kWaves * u;
        const int r = wl * (64 / S::KC) + l / S::KC;
        const int col = swt<S::KC>(r, l % S::KC);
        int64_t key = key0 + (int64_t)b * kFwdBN + r;
        key = key < n_kv ? key : n_kv - 1;
        g2l16(src + ((size_t)key * h_kv + it.g) * D + 8 * col, dst + wl * 512);
      });
    };

    issue(kb0, 0, 0);
    issue(kb0, 0, 1);
    wait_vm();
    __syncthreads();
    for (int b = kb0; b < nkb; ++b) {
      const int buf = (b - kb0) & 1;
      // the next block's K rows after this block's S^T products, its V rows
      // after the softmax (the other workgroup on the CU keeps the matrix
      // cores busy while this one waits to issue; waves without rows in this
      // block post both at once)
      const bool more = b + 1 < nkb;
      if (b >= wave_nkb && more) {
        issue(b + 1, buf ^ 1, 0);
        issue(b + 1, buf ^ 1, 1);
      }
      if (b < wave_nkb) {
        const bf16 *Ks = smem + buf * S::STAGE;
        const bf16 *Vs = Ks + S::K_EL;
        f32x16 s[2];
        static_for<2>([&](auto t) {
          static_for<16>([&](auto r) { s[t][int(r)] = 0.f; });
          const bf16 *kp = Ks + 32 * t * D;
          static_for<D / 16>([&](auto c) {
            s[t] = mfma32(*reinterpret_cast<const bf16x8 *>(kp + koff[c]), qf[c], s[t]);
          });
        });
        if (more) issue(b + 1, buf ^ 1, 0);
        // keys past the row are masked only in blocks that reach past the
        // wave's first row (the diagonal block of each row)
        if (b * kFwdBN + kFwdBN - 1 > wave_qmin) {
          static_for<2>([&](auto t) {
            static_for<16>([&](auto r) {
              const int kl = b * kFwdBN + 32 * t + 16 * (r >> 3) + 8 * kg + (r & 7);
              if (kl > qloc) s[t][int(r)] = -INFINITY;
            });
          });
        }
        // P with the running max.  The block's row sum of P (needed anyway)
        // bounds every P of the row, so the running max only has to move
        // when that sum exceeds 256 (every P then stays <= 256, as with a
        // max test); the first block always sets it.  Only then is the
        // block's row max computed, the row rescaled and P recomputed.
        bf16x8 pf[4];
        float ps = 0.f;
        auto expo = [&](float neg_m) {
          ps = 0.f;
          static_for<2>([&](auto t) {
            static_for<16>([&](auto r) {
              const float p = fast_exp2(__builtin_fmaf(s[t][int(r)], c2, neg_m));
              ps += p;
              pf[2 * t + (r >> 3)][r & 7] = static_cast<bf16>(p);
            });
          });
        };
        bool move = true;
        if (b > kb0) {
          expo(-m_run);
          move = !(row_sum2(ps) <= 256.f);
        }
        if (__builtin_amdgcn_ballot_w64(move)) {
          float mx = -INFINITY;
          static_for<2>([&](auto t) {
            static_for<16>([&](auto r) { mx = fmaxf(mx, s[t][int(r)]); });
          });
          mx = row_max2(mx) * c2;
          const float alpha = move ? fast_exp2(m_run - mx) : 1.f;
          m_run = move ? mx : m_run;
          l_run *= alpha;
          static_for<D / 32>([&](auto dt) {
            static_for<16>([&](auto r) { oacc[dt][int(r)] *= alpha; });
          });
          expo(-m_run);
        }
        l_run += ps;
        if (more) issue(b + 1, buf ^ 1, 1);
        // O^T += V^T P^T; key chunk c = 16 keys from tile row 16 c
        static_for<D / 32>([&](auto dt) {
          static_for<4>([&](auto c) {
            const bf16 *base = Vs + 16 * c * D;
            oacc[dt] = mfma32(lds_tr16x2(base + troff[dt][0], base + troff[dt][1]), pf[c],
                              oacc[dt]);
          });
        });
      }
      wait_vm();
      __syncthreads();
    }

    if (active && it.slot >= 0) {
      // a part of a split item: unnormalised O, the running max and the row
      // sum into its partial slot (rows w * 32 + ln), merged by
      // fwd_combine_kernel
      const float l_tot = row_sum2(l_run);
      if (ln < wrows) {
        float *rec = parts + (size_t)it.slot * fwd_part_floats(D);
        float *op = rec + (size_t)(w * kRows + ln) * D + 8 * kg;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            float4 *dst = reinterpret_cast<float4 *>(op + 32 * dt + 16 * hh);
            dst[0] = make_float4(oacc[dt][8 * hh], oacc[dt][8 * hh + 1], oacc[dt][8 * hh + 2],
                                 oacc[dt][8 * hh + 3]);
            dst[1] = make_float4(oacc[dt][8 * hh + 4], oacc[dt][8 * hh + 5],
                                 oacc[dt][8 * hh + 6], oacc[dt][8 * hh + 7]);
          }
        if (kg == 0) {
          rec[(size_t)kFwdPartRows * D + w * kRows + ln] = m_run;
          rec[(size_t)kFwdPartRows * D + kFwdPartRows + w * kRows + ln] = l_tot;
        }
      }
    } else if (active) {
      const float l_tot = row_sum2(l_run);
      const float inv = 1.f / l_tot;
      if (ln < wrows) {
        bf16 *op = o + ((size_t)row * h_q + head) * D + 8 * kg;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            bf16x8 ov;
#pragma unroll
            for (int i = 0; i < 8; ++i) ov[i] = static_cast<bf16>(oacc[dt][8 * hh + i] * inv);
            *reinterpret_cast<bf16x8 *>(op + 32 * dt + 16 * hh) = ov;
          }
        if (kg == 0) lse[(size_t)head * n_q + row] = (m_run + __builtin_amdgcn_logf(l_tot)) * kLn2;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Host launcher.  `ws` is laid out as: header | items.
static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

int64_t fwd_max_items(int64_t T, int64_t n, int64_t n_q, int h_q, int h_kv) {
  // items <= rows*heads/64 (an item covers >= 64 (row, head) pairs or ends a
  // fragment) + fragments * head chunks.
  // A split item's parts take its place: kFwdSplitSlots of them at most.
  const int64_t frags = T + (int64_t)h_q * n;
  return n_q * (int64_t)h_q / 64 + frags * (int64_t)(h_kv + h_q / 4 + 1) + 1 + kFwdSplitSlots;
}

FwdLayout fwd_layout(int64_t T, int64_t n, int64_t n_q, int64_t n_kv, int h_q, int h_kv, int d,
                     bool split) {
  FwdLayout L;
  L.max_items = fwd_max_items(T, n, n_q, h_q, h_kv);
  L.hdr = 0;
  L.items = align256(kHdrSlots * sizeof(int32_t));
  L.splits = align256(L.items + (size_t)L.max_items * sizeof(FwdItem));
  L.max_parts = split ? kFwdSplitSlots : 0;
  // a split item has at least two parts
  L.parts = align256(L.splits + (size_t)(L.max_parts / 2) * sizeof(FwdSplit));
  L.total = align256(L.parts + (size_t)L.max_parts * fwd_part_floats(d) * sizeof(float));
  return L;
}

template <int D>
static int launch_fwd_d(const bf16 *q, const bf16 *k, const bf16 *v, const int64_t *cu,
                        int64_t n, const libra_tile_t *tiles, int64_t T, int64_t n_q,
                        int64_t n_kv, int h_q, int h_kv, float scale, bf16 *o, float *lse,
                        char *ws, const FwdLayout &L, hipStream_t st, const KernelTimer *tm) {
  int32_t *hdr = reinterpret_cast<int32_t *>(ws + L.hdr);
  FwdItem *items = reinterpret_cast<FwdItem *>(ws + L.items);
  auto *splits = reinterpret_cast<FwdSplit *>(ws + L.splits);
  float *parts = reinterpret_cast<float *>(ws + L.parts);
  static bool attr_set = false;
  if (!attr_set) {
    if (hipFuncSetAttribute(reinterpret_cast<const void *>(&attn_fwd_kernel<D>),
                            hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)FwdShape<D>::SMEM) != hipSuccess)
      return fail(LIBRA_EHIP, "hipFuncSetAttribute failed");
    attr_set = true;
  }
  int dev = 0, cus = 256;
  hipGetDevice(&dev);
  hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  const int grid = cus * 2;
  hipLaunchKernelGGL(prep_fwd_kernel, dim3(1), dim3(kPrepThreads), 0, st, cu, n, tiles, T, h_q,
                     h_kv, n_q, n_kv, hdr, items, L.max_items, 1, grid, L.max_parts, 0, splits);
  if (tm) hipEventRecord(tm->begin, st);
  hipLaunchKernelGGL(attn_fwd_kernel<D>, dim3(grid), dim3(kThreads), FwdShape<D>::SMEM, st, q,
                     k, v, cu, items, hdr, h_q, h_kv, n_q, n_kv, scale * kLog2e, o,
                     lse, parts);
  if (L.max_parts > 0)
    hipLaunchKernelGGL(fwd_combine_kernel<D>, dim3(cus), dim3(256), 0, st, splits, hdr, parts,
                       h_q, n_q, o, lse);
  if (tm) hipEventRecord(tm->end, st);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(LIBRA_EHIP, "forward launch failed: %s", hipGetErrorString(e));
  return LIBRA_OK;
}

void enqueue_fwd_items(const int64_t *cu, int64_t n, const libra_tile_t *tiles, int64_t T,
                       int h_q, int h_kv, int64_t n_q, int64_t n_kv, int32_t *hdr,
                       FwdItem *items, int64_t max_items, bool count_bad, int grid,
                       int max_parts, FwdSplit *splits, hipStream_t st) {
  hipLaunchKernelGGL(prep_fwd_kernel, dim3(1), dim3(kPrepThreads), 0, st, cu, n, tiles, T, h_q,
                     h_kv, n_q, n_kv, hdr, items, max_items, count_bad ? 1 : 0, grid, max_parts,
                     1, splits);
}

int launch_fwd(const void *q, const void *k, const void *v, const int64_t *cu, int64_t n,
               const libra_tile_t *tiles, int64_t T, int64_t n_q, int64_t n_kv, int h_q,
               int h_kv, int d, float scale, void *o, float *lse, void *ws,
               const FwdLayout &L, hipStream_t st, const KernelTimer *tm) {
  auto Q = static_cast<const bf16 *>(q);
  auto K = static_cast<const bf16 *>(k);
  auto V = static_cast<const bf16 *>(v);
  auto O = static_cast<bf16 *>(o);
  char *W = static_cast<char *>(ws);
  if (d == 128)
    return launch_fwd_d<128>(Q, K, V, cu, n, tiles, T, n_q, n_kv, h_q, h_kv, scale, O, lse, W, L,
                             st, tm);
  return launch_fwd_d<64>(Q, K, V, cu, n, tiles, T, n_q, n_kv, h_q, h_kv, scale, O, lse, W, L, st,
                          tm);
}

}  // namespace libra
