// Forward pass of document-masked causal attention over SH-Tiles (gfx950).
//
// What is computed: Eq. 1 of the paper under the block-diagonal causal mask of
// packing (Sec. 2.3), for the (row, query head) pairs covered by a list of
// SH-Tiles (Sec. 4.3.1).  Each tile is cut into work items on the device; a
// persistent kernel walks the items longest-first.
//
// Kernel structure (one work item = up to 4 query heads of one KV group x 32
// rows per head, or fewer heads x more rows; 4 waves, one (head, 32 rows) each):
//   * K blocks of 64 keys and the matching V^T block are staged in LDS,
//     double-buffered; blocks are anchored at the sample start and only the
//     row's own sample is visited, so cross-document blocks are never touched.
//   * S^T = K Q^T with v_mfma_f32_32x32x16_bf16 (keys on M, queries on N), so
//     that every lane owns one query: the row max / row sum of the online
//     softmax are 32 in-lane values plus one exchange with lane ^ 32.
//   * O^T += V^T P^T with the same instruction; P^T comes straight from the
//     S^T accumulators (bf16), V^T from a transposed copy of V laid out with
//     every sample starting on a 64-key boundary (zero padded).
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "attn_common.h"
#include "errors.h"

namespace libra {

// ---------------------------------------------------------------------------
// Work items: every tile is split into sample fragments; every fragment into
// items of (<= 4 heads of one KV group) x (32 * 4 / heads rows).
template <typename F>
__device__ void for_each_fwd_item(const libra_tile_t &t, const int64_t *cu, int64_t n, int G,
                                  F &&f) {
  int64_t j = upper_bound64(cu, n, t.q_begin) - 1;
  for (; j < n && cu[j] < t.q_end; ++j) {
    const int64_t pb = t.q_begin > cu[j] ? t.q_begin : cu[j];
    const int64_t pe = t.q_end < cu[j + 1] ? t.q_end : cu[j + 1];
    const int32_t row0 = (int32_t)(t.q_row + (pb - t.q_begin));
    const int32_t qloc0 = (int32_t)(pb - cu[j]);
    const int32_t nfrag = (int32_t)(pe - pb);
    for (int g = t.head_begin / G; g * G < t.head_end; ++g) {
      const int hl = max(t.head_begin, g * G), hh = min(t.head_end, (g + 1) * G);
      for (int h0 = hl; h0 < hh; h0 += 4) {
        const int nh = min(4, hh - h0);
        const int rows_per = kRows * (4 / nh);
        for (int rb = 0; rb < nfrag; rb += rows_per) {
          const int nrows = min(rows_per, nfrag - rb);
          FwdItem it{row0 + rb, qloc0 + rb, (int32_t)j, h0, nh, nrows, g, 0};
          f(it, (qloc0 + rb + nrows - 1) / kFwdBN + 1);
        }
      }
    }
  }
}

// One workgroup: count items per cost bucket, order buckets longest-first,
// scatter.  Also resets the queue.  Tiles outside the buffers are skipped and
// counted in hdr[kBadTiles].
__global__ __launch_bounds__(kPrepThreads) void prep_fwd_kernel(
    const int64_t *__restrict__ cu, int64_t n, const libra_tile_t *__restrict__ tiles, int64_t T,
    int h_q, int h_kv, int64_t n_q, int64_t n_kv, int32_t *__restrict__ hdr,
    FwdItem *__restrict__ items, int64_t max_items) {
  __shared__ int32_t hist[kBuckets];
  __shared__ int32_t part[kPrepThreads];
  __shared__ int32_t bad;
  const int tid = threadIdx.x;
  const int G = h_q / h_kv;
  for (int i = tid; i < kBuckets; i += kPrepThreads) hist[i] = 0;
  if (tid == 0) bad = 0;
  __syncthreads();
  auto bucket = [](int nkb) { return kBuckets - (nkb < kBuckets ? nkb : kBuckets); };
  for (int64_t t = tid; t < T; t += kPrepThreads) {
    const libra_tile_t tl = tiles[t];
    if (!tile_ok(tl, n_q, n_kv, h_q)) { atomicAdd(&bad, 1); continue; }
    for_each_fwd_item(tl, cu, n, G, [&](const FwdItem &, int nkb) {
      atomicAdd(&hist[bucket(nkb)], 1);
    });
  }
  __syncthreads();
  // exclusive scan over buckets (bucket 0 = longest)
  constexpr int per = kBuckets / kPrepThreads;
  int32_t s = 0;
  for (int i = 0; i < per; ++i) s += hist[tid * per + i];
  part[tid] = s;
  __syncthreads();
  for (int o = 1; o < kPrepThreads; o <<= 1) {
    const int32_t v = tid >= o ? part[tid - o] : 0;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  int32_t base = part[tid] - s;
  const int32_t total = part[kPrepThreads - 1];
  __syncthreads();
  for (int i = 0; i < per; ++i) {
    const int32_t c = hist[tid * per + i];
    hist[tid * per + i] = base;
    base += c;
  }
  __syncthreads();
  for (int64_t t = tid; t < T; t += kPrepThreads) {
    const libra_tile_t tl = tiles[t];
    if (!tile_ok(tl, n_q, n_kv, h_q)) continue;
    for_each_fwd_item(tl, cu, n, G, [&](const FwdItem &it, int nkb) {
      const int32_t pos = atomicAdd(&hist[bucket(nkb)], 1);
      if (pos < max_items) items[pos] = it;
    });
  }
  if (tid == 0) {
    hdr[kFwdQueue] = 0;
    hdr[kFwdItems] = total < max_items ? total : (int32_t)max_items;
    hdr[kBadTiles] = bad + (total > max_items ? 1 : 0);
  }
}

// ---------------------------------------------------------------------------
// V [n_kv][h_kv][D] -> Vt [h_kv][D][pitch]; sample j occupies
// [vt_offset(cu[j], j), +ceil64(len)), zero padded past its length.
template <int D>
__global__ __launch_bounds__(256) void transpose_v_kernel(const bf16 *__restrict__ v,
                                                          const int64_t *__restrict__ cu,
                                                          int64_t n, int64_t n_kv, int h_kv,
                                                          int64_t pitch, bf16 *__restrict__ vt) {
  __shared__ bf16 tile[64][D + 2];
  __shared__ int64_t pos[64];
  __shared__ int32_t pad_len[64];
  const int g = blockIdx.y;
  const int64_t k0 = (int64_t)blockIdx.x * 64;
  const int tid = threadIdx.x;
  for (int ci = tid; ci < 64 * D / 2; ci += 256) {
    const int r = ci / (D / 2), c2 = ci % (D / 2);
    const int64_t key = k0 + r;
    uint32_t val = 0;
    if (key < n_kv)
      val = *reinterpret_cast<const uint32_t *>(v + ((size_t)key * h_kv + g) * D + 2 * c2);
    *reinterpret_cast<uint32_t *>(&tile[r][2 * c2]) = val;
  }
  if (tid < 64) {
    const int64_t key = k0 + tid;
    pos[tid] = -1;
    pad_len[tid] = 0;
    if (key < n_kv) {
      const int64_t j = upper_bound64(cu, n, key) - 1;
      const int64_t len = cu[j + 1] - cu[j];
      pos[tid] = vt_offset(cu[j], j) + (key - cu[j]);
      if (key + 1 == cu[j + 1]) pad_len[tid] = (int32_t)((len + 63) / 64 * 64 - len);
    }
  }
  __syncthreads();
  for (int e = tid; e < 64 * D; e += 256) {
    const int dd = e / 64, r = e % 64;
    if (pos[r] >= 0) vt[((size_t)g * D + dd) * pitch + pos[r]] = tile[r][dd];
  }
  for (int r = 0; r < 64; ++r) {
    if (pad_len[r] == 0) continue;
    for (int e = tid; e < 64 * D; e += 256) {
      const int dd = e / 64, p = e % 64;
      if (p < pad_len[r]) vt[((size_t)g * D + dd) * pitch + pos[r] + 1 + p] = bf16(0.0f);
    }
  }
}

// ---------------------------------------------------------------------------
template <int D>
struct FwdShape {
  static constexpr int KP = D + 8;            // K tile pitch (elements)
  static constexpr int VP = kFwdBN + 8;       // V^T tile pitch
  static constexpr int K_EL = kFwdBN * KP;
  static constexpr int V_EL = D * VP;
  static constexpr int STAGE = K_EL + V_EL;
  static constexpr int NK = kFwdBN * D / 8 / kThreads;   // 16-byte K loads per thread
  static constexpr int NV = D * kFwdBN / 8 / kThreads;   // 16-byte V^T loads per thread
  static constexpr size_t SMEM = 2 * STAGE * sizeof(bf16);
};

template <int D>
__global__ __launch_bounds__(kThreads, 2) void attn_fwd_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ k, const bf16 *__restrict__ vt,
    const int64_t *__restrict__ cu, const FwdItem *__restrict__ items, int32_t *__restrict__ hdr,
    int h_q, int h_kv, int64_t n_q, int64_t n_kv, int64_t pitch, float c2,
    bf16 *__restrict__ o, float *__restrict__ lse) {
  using S = FwdShape<D>;
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  __shared__ int32_t s_item;
  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, ln = l & 31, kg = l >> 5;
  const int n_items = hdr[kFwdItems];

  for (;;) {
    if (tid == 0) s_item = atomicAdd(&hdr[kFwdQueue], 1);
    __syncthreads();
    const int idx = s_item;
    if (idx >= n_items) break;
    const FwdItem it = items[idx];
    const int64_t key0 = cu[it.sample];
    const int64_t voff = vt_offset(key0, it.sample);
    const int head = it.head0 + (w % it.nh);
    const int wrow0 = (w / it.nh) * kRows;
    const int wrows = min(max(it.nrows - wrow0, 0), kRows);
    const bool active = wrows > 0;
    const int my_r = active ? min(ln, wrows - 1) : 0;
    const int64_t row = (int64_t)it.q_row0 + wrow0 + my_r;
    const int qloc = it.q_loc0 + wrow0 + my_r;
    const int wave_qmin = it.q_loc0 + wrow0;
    const int nkb = (it.q_loc0 + it.nrows - 1) / kFwdBN + 1;
    const int wave_nkb = active ? (it.q_loc0 + wrow0 + wrows - 1) / kFwdBN + 1 : 0;

    bf16x8 qf[D / 16];
    if (active) {
      const bf16 *qp = q + ((size_t)row * h_q + head) * D + 8 * kg;
#pragma unroll
      for (int c = 0; c < D / 16; ++c) qf[c] = *reinterpret_cast<const bf16x8 *>(qp + 16 * c);
    }
    f32x16 oacc[D / 32];
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[dt][r] = 0.f;
    float m_run = -INFINITY, l_run = 0.f;

    // staging: registers <- global for block b
    uint4 kreg[S::NK], vreg[S::NV];
    auto fetch = [&](int b) {
#pragma unroll
      for (int u = 0; u < S::NK; ++u) {
        const int ci = tid + kThreads * u;
        const int r = ci / (D / 8), c8 = ci % (D / 8);
        const int64_t key = key0 + (int64_t)b * kFwdBN + r;
        kreg[u] = key < n_kv ? *reinterpret_cast<const uint4 *>(
                                   k + ((size_t)key * h_kv + it.g) * D + 8 * c8)
                             : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int u = 0; u < S::NV; ++u) {
        const int ci = tid + kThreads * u;
        const int dd = ci / (kFwdBN / 8), c8 = ci % (kFwdBN / 8);
        vreg[u] = *reinterpret_cast<const uint4 *>(
            vt + ((size_t)it.g * D + dd) * pitch + voff + (int64_t)b * kFwdBN + 8 * c8);
      }
    };
    auto stash = [&](int buf) {
      bf16 *Ks = smem + buf * S::STAGE;
      bf16 *Vs = Ks + S::K_EL;
#pragma unroll
      for (int u = 0; u < S::NK; ++u) {
        const int ci = tid + kThreads * u;
        const int r = ci / (D / 8), c8 = ci % (D / 8);
        *reinterpret_cast<uint4 *>(Ks + r * S::KP + 8 * c8) = kreg[u];
      }
#pragma unroll
      for (int u = 0; u < S::NV; ++u) {
        const int ci = tid + kThreads * u;
        const int dd = ci / (kFwdBN / 8), c8 = ci % (kFwdBN / 8);
        *reinterpret_cast<uint4 *>(Vs + dd * S::VP + 8 * c8) = vreg[u];
      }
    };

    fetch(0);
    stash(0);
    __syncthreads();
    for (int b = 0; b < nkb; ++b) {
      const int buf = b & 1;
      if (b + 1 < nkb) fetch(b + 1);
      if (b < wave_nkb) {
        const bf16 *Ks = smem + buf * S::STAGE;
        const bf16 *Vs = Ks + S::K_EL;
        f32x16 s[2];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
          for (int r = 0; r < 16; ++r) s[t][r] = 0.f;
          const bf16 *kp = Ks + (32 * t + perm32(ln)) * S::KP + 8 * kg;
#pragma unroll
          for (int c = 0; c < D / 16; ++c)
            s[t] = mfma32(*reinterpret_cast<const bf16x8 *>(kp + 16 * c), qf[c], s[t]);
        }
        const bool need_mask = b * kFwdBN + kFwdBN - 1 > wave_qmin;
        float mx = -INFINITY;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            float x = s[t][r] * c2;
            const int kl = b * kFwdBN + 32 * t + 16 * (r >> 3) + 8 * kg + (r & 7);
            if (need_mask && kl > qloc) x = -INFINITY;
            s[t][r] = x;
            mx = fmaxf(mx, x);
          }
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run, mx);
        const float alpha = fast_exp2(m_run - m_new);
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[dt][r] *= alpha;
        bf16x8 pf[4];
        float ps = 0.f;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const float p = fast_exp2(s[t][r] - m_new);
            ps += p;
            pf[2 * t + (r >> 3)][r & 7] = static_cast<bf16>(p);
          }
        l_run += ps;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt) {
          const bf16 *vp = Vs + (32 * dt + perm32(ln)) * S::VP + 8 * kg;
#pragma unroll
          for (int c = 0; c < 4; ++c)
            oacc[dt] = mfma32(*reinterpret_cast<const bf16x8 *>(vp + 16 * c), pf[c], oacc[dt]);
        }
      }
      if (b + 1 < nkb) stash(buf ^ 1);
      __syncthreads();
    }

    if (active) {
      const float l_tot = l_run + __shfl_xor(l_run, 32);
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
// Host launcher.  `ws` is laid out as: header | items | Vt.
static size_t align256(size_t x) { return (x + 255) / 256 * 256; }

FwdLayout fwd_layout(int64_t T, int64_t n, int64_t n_q, int64_t n_kv, int h_q, int h_kv, int d) {
  FwdLayout L;
  // items <= rows*heads/64 (item covers >= 64 (row, head) pairs or ends a
  // fragment) + fragments * head chunks.
  const int64_t frags = T + (int64_t)h_q * n;
  L.max_items = n_q * (int64_t)h_q / 64 + frags * (int64_t)(h_kv + h_q / 4 + 1) + 1;
  L.pitch = vt_pitch(n_kv, n);
  L.hdr = 0;
  L.items = align256(kHdrSlots * sizeof(int32_t));
  L.vt = align256(L.items + (size_t)L.max_items * sizeof(FwdItem));
  L.total = align256(L.vt + (size_t)h_kv * d * L.pitch * sizeof(bf16));
  return L;
}

template <int D>
static int launch_fwd_d(const bf16 *q, const bf16 *k, const bf16 *v, const int64_t *cu,
                        int64_t n, const libra_tile_t *tiles, int64_t T, int64_t n_q,
                        int64_t n_kv, int h_q, int h_kv, float scale, bf16 *o, float *lse,
                        char *ws, const FwdLayout &L, hipStream_t st, const KernelTimer *tm) {
  int32_t *hdr = reinterpret_cast<int32_t *>(ws + L.hdr);
  FwdItem *items = reinterpret_cast<FwdItem *>(ws + L.items);
  bf16 *vt = reinterpret_cast<bf16 *>(ws + L.vt);
  static bool attr_set = false;
  if (!attr_set) {
    if (hipFuncSetAttribute(reinterpret_cast<const void *>(&attn_fwd_kernel<D>),
                            hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)FwdShape<D>::SMEM) != hipSuccess)
      return fail(LIBRA_EHIP, "hipFuncSetAttribute failed");
    attr_set = true;
  }
  hipLaunchKernelGGL(prep_fwd_kernel, dim3(1), dim3(kPrepThreads), 0, st, cu, n, tiles, T, h_q,
                     h_kv, n_q, n_kv, hdr, items, L.max_items);
  hipLaunchKernelGGL(transpose_v_kernel<D>, dim3((unsigned)((n_kv + 63) / 64), h_kv), dim3(256),
                     0, st, v, cu, n, n_kv, h_kv, L.pitch, vt);
  int dev = 0, cus = 256;
  hipGetDevice(&dev);
  hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (tm) hipEventRecord(tm->begin, st);
  hipLaunchKernelGGL(attn_fwd_kernel<D>, dim3(cus * 2), dim3(kThreads), FwdShape<D>::SMEM, st, q,
                     k, vt, cu, items, hdr, h_q, h_kv, n_q, n_kv, L.pitch, scale * kLog2e, o,
                     lse);
  if (tm) hipEventRecord(tm->end, st);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(LIBRA_EHIP, "forward launch failed: %s", hipGetErrorString(e));
  return LIBRA_OK;
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
