// Backward pass of document-masked causal attention over SH-Tiles (gfx950).
//
// Textbook attention gradients (the paper's backward reuses the forward
// assignment with reversed transfers, Sec. 4.3.3, so it computes exactly
// these): P = exp(S - LSE), D = rowsum(dO * O), dV = P^T dO,
// dS = P * (dO V^T - D), dQ = scale dS K, dK = scale dS^T Q.
//
// Structure:
//   * a pre-pass writes D, transposed copies Q^T / dO^T of the covered rows
//     (so every MFMA operand is read from LDS as 16 contiguous bytes) and
//     clears the fp32 dQ accumulator;
//   * one workgroup prepares KV-block work items, longest-first;
//   * a persistent KV-stationary kernel: a work item is 128 keys of one KV
//     head of one sample (anchored at the sample start); each of the 4 waves
//     keeps 32 keys of K and V in registers plus fp32 dK^T / dV^T
//     accumulators, and loops over the 32-row query blocks of the tiles that
//     attend them and over the query heads of the KV group.  S and dP are
//     computed with queries on M (lane = key), which is exactly the operand
//     layout dV^T = dO^T P and dK^T = Q^T dS need; dS goes through LDS once
//     so that dQ = dS K over all 128 keys is one contraction per wave,
//     accumulated into fp32 with hardware float atomics;
//   * a finalize pass converts dQ to bf16 for the covered rows and heads.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "attn_common.h"
#include "errors.h"

namespace libra {

__device__ __forceinline__ int32_t ld_agent(const int32_t *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long ld_agent(const unsigned long long *p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Bit set of the KV heads whose query groups intersect [hb, he).
__device__ __forceinline__ unsigned long long group_bits(int hb, int he, int G) {
  unsigned long long m = 0;
  for (int g = hb / G; g * G < he; ++g) m |= 1ull << g;
  return m;
}

// ---------------------------------------------------------------------------
// One workgroup: per sample, the key extent attended by covered rows and the
// KV heads involved; then items (sample, 128-key block, KV head) ordered by
// the number of attending rows, longest first.
__global__ __launch_bounds__(kPrepThreads) void prep_bwd_kernel(
    const int64_t *__restrict__ cu, int64_t n, const libra_tile_t *__restrict__ tiles, int64_t T,
    int h_q, int h_kv, int64_t n_q, int64_t n_kv, int32_t *__restrict__ hdr,
    int32_t *__restrict__ ext, unsigned long long *__restrict__ gmask,
    BwdItem *__restrict__ items, int64_t max_items) {
  __shared__ int32_t hist[kBuckets];
  __shared__ int32_t part[kPrepThreads];
  __shared__ int32_t bad;
  const int tid = threadIdx.x;
  const int G = h_q / h_kv;
  for (int64_t j = tid; j < n; j += kPrepThreads) {
    __hip_atomic_store(&ext[j], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_store(&gmask[j], 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  for (int i = tid; i < kBuckets; i += kPrepThreads) hist[i] = 0;
  if (tid == 0) bad = 0;
  __threadfence();
  __syncthreads();
  for (int64_t t = tid; t < T; t += kPrepThreads) {
    const libra_tile_t tl = tiles[t];
    if (!tile_ok(tl, n_q, n_kv, h_q)) { atomicAdd(&bad, 1); continue; }
    const unsigned long long bits = group_bits(tl.head_begin, tl.head_end, G);
    for (int64_t j = upper_bound64(cu, n, tl.q_begin) - 1; j < n && cu[j] < tl.q_end; ++j) {
      const int64_t pe = tl.q_end < cu[j + 1] ? tl.q_end : cu[j + 1];
      atomicMax(&ext[j], (int32_t)(pe - cu[j]));
      atomicOr(&gmask[j], bits);
    }
  }
  __threadfence();
  __syncthreads();
  auto bucket = [](int32_t e, int kb) {
    const int32_t c = (e - kb * kBwdBK + kRows - 1) / kRows;   // attending row blocks
    return kBuckets - (c < kBuckets ? c : kBuckets);
  };
  for (int64_t j = tid; j < n; j += kPrepThreads) {
    const int32_t e = ld_agent(&ext[j]);
    if (e == 0) continue;
    const unsigned long long mk = ld_agent(&gmask[j]);
    const int nkb = (e + kBwdBK - 1) / kBwdBK;
    for (int g = 0; g < h_kv; ++g)
      if (mk >> g & 1ull)
        for (int kb = 0; kb < nkb; ++kb) atomicAdd(&hist[bucket(e, kb)], 1);
  }
  __syncthreads();
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
  for (int64_t j = tid; j < n; j += kPrepThreads) {
    const int32_t e = ld_agent(&ext[j]);
    if (e == 0) continue;
    const unsigned long long mk = ld_agent(&gmask[j]);
    const int nkb = (e + kBwdBK - 1) / kBwdBK;
    for (int g = 0; g < h_kv; ++g)
      if (mk >> g & 1ull)
        for (int kb = 0; kb < nkb; ++kb) {
          const int32_t pos = atomicAdd(&hist[bucket(e, kb)], 1);
          if (pos < max_items) items[pos] = BwdItem{(int32_t)j, kb, g, 0};
        }
  }
  if (tid == 0) {
    hdr[kBwdQueue] = 0;
    hdr[kBwdItems] = total < max_items ? total : (int32_t)max_items;
    hdr[kBadTiles] = bad + (total > max_items ? 1 : 0);
  }
}

// ---------------------------------------------------------------------------
// Pre-pass over the covered (row, head) pairs, 32 rows at a time:
// D = rowsum(dO * O), Q^T and dO^T as [h_q][D][nq_pad], dQ accumulator = 0.
constexpr int kTileSplit = 64;

template <int D>
__global__ __launch_bounds__(256) void bwd_pre_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ o, const bf16 *__restrict__ dout,
    const libra_tile_t *__restrict__ tiles, int h_q, int64_t n_q, int64_t n_kv, int64_t nq_pad,
    float *__restrict__ dvec, bf16 *__restrict__ qt, bf16 *__restrict__ dot,
    float *__restrict__ dqacc) {
  __shared__ bf16 tq[kRows][D + 2];
  __shared__ bf16 tdo[kRows][D + 2];
  const int tid = threadIdx.x;
  const libra_tile_t tl = tiles[blockIdx.x / kTileSplit];
  if (!tile_ok(tl, n_q, n_kv, h_q)) return;
  const int64_t ra = tl.q_row, rb = tl.q_row + (tl.q_end - tl.q_begin);
  for (int64_t m = ra / kRows + blockIdx.x % kTileSplit; m * kRows < rb; m += kTileSplit) {
    const int64_t lo = m * kRows > ra ? m * kRows : ra;
    const int64_t hi = (m + 1) * kRows < rb ? (m + 1) * kRows : rb;
    for (int h = tl.head_begin; h < tl.head_end; ++h) {
      for (int ci = tid; ci < kRows * D / 2; ci += 256) {
        const int r = ci / (D / 2), c2 = ci % (D / 2);
        const int64_t row = m * kRows + r;
        uint32_t qv = 0, dv = 0;
        if (row >= lo && row < hi) {
          const size_t off = ((size_t)row * h_q + h) * D + 2 * c2;
          qv = *reinterpret_cast<const uint32_t *>(q + off);
          dv = *reinterpret_cast<const uint32_t *>(dout + off);
        }
        *reinterpret_cast<uint32_t *>(&tq[r][2 * c2]) = qv;
        *reinterpret_cast<uint32_t *>(&tdo[r][2 * c2]) = dv;
      }
      {
        const int r = tid >> 3, part = tid & 7;
        const int64_t row = m * kRows + r;
        float acc = 0.f;
        if (row >= lo && row < hi) {
          const size_t off = ((size_t)row * h_q + h) * D + part * (D / 8);
#pragma unroll
          for (int i = 0; i < D / 8; ++i)
            acc += static_cast<float>(o[off + i]) * static_cast<float>(dout[off + i]);
        }
        acc += __shfl_xor(acc, 1);
        acc += __shfl_xor(acc, 2);
        acc += __shfl_xor(acc, 4);
        if (part == 0 && row >= lo && row < hi) dvec[(size_t)h * n_q + row] = acc;
      }
      for (int ci = tid; ci < kRows * D / 4; ci += 256) {
        const int r = ci / (D / 4), c4 = ci % (D / 4);
        const int64_t row = m * kRows + r;
        if (row >= lo && row < hi)
          *reinterpret_cast<float4 *>(dqacc + ((size_t)row * h_q + h) * D + 4 * c4) =
              make_float4(0.f, 0.f, 0.f, 0.f);
      }
      __syncthreads();
      for (int e = tid; e < D * kRows; e += 256) {
        const int dd = e / kRows, r = e % kRows;
        const int64_t row = m * kRows + r;
        if (row >= lo && row < hi) {
          const size_t off = ((size_t)h * D + dd) * nq_pad + row;
          qt[off] = tq[r][dd];
          dot[off] = tdo[r][dd];
        }
      }
      __syncthreads();
    }
  }
}

// dQ (bf16) <- fp32 accumulator for the covered (row, head) pairs.
template <int D>
__global__ __launch_bounds__(256) void bwd_finalize_kernel(const libra_tile_t *__restrict__ tiles,
                                                           int h_q, int64_t n_q, int64_t n_kv,
                                                           const float *__restrict__ dqacc,
                                                           bf16 *__restrict__ dq) {
  const libra_tile_t tl = tiles[blockIdx.x / kTileSplit];
  if (!tile_ok(tl, n_q, n_kv, h_q)) return;
  const int64_t ra = tl.q_row, rb = tl.q_row + (tl.q_end - tl.q_begin);
  const int nh = tl.head_end - tl.head_begin;
  const int64_t per_row = (int64_t)nh * D / 8;       // 8-element groups per row
  const int64_t total = (rb - ra) * per_row;
  for (int64_t e = (int64_t)(blockIdx.x % kTileSplit) * 256 + threadIdx.x; e < total;
       e += (int64_t)kTileSplit * 256) {
    const int64_t row = ra + e / per_row;
    const int64_t rem = e % per_row;
    const int h = tl.head_begin + (int)(rem / (D / 8));
    const int c8 = (int)(rem % (D / 8));
    const size_t off = ((size_t)row * h_q + h) * D + 8 * c8;
    const float4 a = *reinterpret_cast<const float4 *>(dqacc + off);
    const float4 b = *reinterpret_cast<const float4 *>(dqacc + off + 4);
    bf16x8 v;
    v[0] = static_cast<bf16>(a.x); v[1] = static_cast<bf16>(a.y);
    v[2] = static_cast<bf16>(a.z); v[3] = static_cast<bf16>(a.w);
    v[4] = static_cast<bf16>(b.x); v[5] = static_cast<bf16>(b.y);
    v[6] = static_cast<bf16>(b.z); v[7] = static_cast<bf16>(b.w);
    *reinterpret_cast<bf16x8 *>(dq + off) = v;
  }
}

__global__ __launch_bounds__(256) void zero_kernel(uint4 *__restrict__ p, int64_t n16) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n16;
       i += (int64_t)gridDim.x * 256)
    p[i] = make_uint4(0, 0, 0, 0);
}

// ---------------------------------------------------------------------------
template <int D>
struct BwdShape {
  static constexpr int QP = D + 8;          // Q / dO tile pitch (row-major, 32 rows)
  static constexpr int TP = kRows + 8;      // Q^T / dO^T tile pitch (D rows)
  static constexpr int SP = kBwdBK + 8;     // dS tile pitch (32 rows x 128 keys)
  static constexpr int KP = D + 8;          // K block pitch (128 rows), setup only
  static constexpr int Q_EL = kRows * QP;
  static constexpr int T_EL = D * TP;
  static constexpr int STAGE_EL = 2 * Q_EL + 2 * T_EL;
  static constexpr int S_EL = kRows * SP;
  static constexpr int K_EL = kBwdBK * KP;
  static constexpr int MAIN_EL = STAGE_EL + S_EL;
  static constexpr int BF_EL = MAIN_EL > K_EL ? MAIN_EL : K_EL;
  static constexpr size_t SMEM = BF_EL * sizeof(bf16) + 2 * kRows * sizeof(float);
  // dQ split: D=128 -> wave w owns d-tile w over all 8 key chunks;
  //           D=64  -> wave w owns d-tile w&1 over key chunks 4*(w>>1)..+3.
  static constexpr int DQ_CHUNKS = D == 128 ? 8 : 4;
};

template <int D>
__global__ __launch_bounds__(kThreads, 1) void attn_bwd_kernel(
    const bf16 *__restrict__ k, const bf16 *__restrict__ v, const bf16 *__restrict__ q,
    const bf16 *__restrict__ dout, const bf16 *__restrict__ qt, const bf16 *__restrict__ dot,
    const float *__restrict__ lse, const float *__restrict__ dvec,
    const int64_t *__restrict__ cu, const libra_tile_t *__restrict__ tiles, int64_t T,
    const BwdItem *__restrict__ items, int32_t *__restrict__ hdr, int h_q, int h_kv,
    int64_t n_q, int64_t n_kv, int64_t nq_pad, float scale, float c2,
    float *__restrict__ dqacc, void *__restrict__ dk_out, void *__restrict__ dv_out,
    int accumulate) {
  using S = BwdShape<D>;
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  bf16 *Qs = smem;
  bf16 *dOs = Qs + S::Q_EL;
  bf16 *Qts = dOs + S::Q_EL;
  bf16 *dOts = Qts + S::T_EL;
  bf16 *Ss = dOts + S::T_EL;
  bf16 *Ks = smem;                                   // aliases the above during setup
  float *lse2s = reinterpret_cast<float *>(smem + S::BF_EL);
  float *dvs = lse2s + kRows;
  __shared__ int32_t s_item;

  const int tid = threadIdx.x, w = tid >> 6, l = tid & 63, ln = l & 31, kg = l >> 5;
  const int G = h_q / h_kv;
  const int n_items = hdr[kBwdItems];
  const int dq_dt = D == 128 ? w : (w & 1);
  const int dq_c0 = D == 128 ? 0 : 4 * (w >> 1);

  for (;;) {
    if (tid == 0) s_item = atomicAdd(&hdr[kBwdQueue], 1);
    __syncthreads();
    const int idx = s_item;
    if (idx >= n_items) break;
    const BwdItem it = items[idx];
    const int64_t key0 = cu[it.sample];
    const int64_t len = cu[it.sample + 1] - key0;
    const int g = it.g;
    const int kloc0 = it.kb * kBwdBK;                 // first key of the block (sample-local)
    const int kl = kloc0 + 32 * w + ln;               // this lane's key
    const bool key_ok = kl < len;
    const int64_t krow = key0 + kl;

    bf16x8 kf[D / 16], vf[D / 16];
#pragma unroll
    for (int c = 0; c < D / 16; ++c) {
      if (key_ok) {
        const size_t off = ((size_t)krow * h_kv + g) * D + 16 * c + 8 * kg;
        kf[c] = *reinterpret_cast<const bf16x8 *>(k + off);
        vf[c] = *reinterpret_cast<const bf16x8 *>(v + off);
      } else {
#pragma unroll
        for (int i = 0; i < 8; ++i) { kf[c][i] = bf16(0.f); vf[c][i] = bf16(0.f); }
      }
      *reinterpret_cast<bf16x8 *>(Ks + (32 * w + ln) * S::KP + 16 * c + 8 * kg) = kf[c];
    }
    __syncthreads();
    // K fragments for dQ = dS K: B operand, lane = d column, 8 consecutive keys.
    bf16x8 kq[S::DQ_CHUNKS];
#pragma unroll
    for (int c = 0; c < S::DQ_CHUNKS; ++c)
#pragma unroll
      for (int i = 0; i < 8; ++i)
        kq[c][i] = Ks[(16 * (dq_c0 + c) + 8 * kg + i) * S::KP + 32 * dq_dt + ln];
    __syncthreads();

    f32x16 dva[D / 32], dka[D / 32];
#pragma unroll
    for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
      for (int r = 0; r < 16; ++r) { dva[dt][r] = 0.f; dka[dt][r] = 0.f; }

    for (int64_t t = 0; t < T; ++t) {
      const libra_tile_t tl = tiles[t];
      if (!tile_ok(tl, n_q, n_kv, h_q)) continue;
      const int64_t pb = tl.q_begin > key0 ? tl.q_begin : key0;
      const int64_t pe = tl.q_end < key0 + len ? tl.q_end : key0 + len;
      if (pb >= pe) continue;
      const int h0 = max(tl.head_begin, g * G), h1 = min(tl.head_end, (g + 1) * G);
      if (h0 >= h1) continue;
      const int64_t fra = tl.q_row + (pb - tl.q_begin);   // fragment rows [fra, frb)
      const int64_t frb = fra + (pe - pb);
      const int64_t qla = pb - key0;                      // sample-local position of fra
      const int64_t first = fra + (kloc0 > qla ? kloc0 - qla : 0);
      if (first >= frb) continue;
      for (int64_t m = first / kRows; m * kRows < frb; ++m) {
        const int64_t lo = m * kRows > fra ? m * kRows : fra;
        const int64_t hi = (m + 1) * kRows < frb ? (m + 1) * kRows : frb;
        for (int h = h0; h < h1; ++h) {
          // ---- stage the 32-row query block of head h
          for (int ci = tid; ci < kRows * D / 8; ci += kThreads) {
            const int r = ci / (D / 8), c8 = ci % (D / 8);
            const int64_t row = m * kRows + r;
            uint4 a = make_uint4(0, 0, 0, 0), b = a;
            if (row >= lo && row < hi) {
              const size_t off = ((size_t)row * h_q + h) * D + 8 * c8;
              a = *reinterpret_cast<const uint4 *>(q + off);
              b = *reinterpret_cast<const uint4 *>(dout + off);
            }
            *reinterpret_cast<uint4 *>(Qs + r * S::QP + 8 * c8) = a;
            *reinterpret_cast<uint4 *>(dOs + r * S::QP + 8 * c8) = b;
          }
          for (int ci = tid; ci < D * kRows / 8; ci += kThreads) {
            const int dd = ci / (kRows / 8), c8 = ci % (kRows / 8);
            const int64_t row0 = m * kRows + 8 * c8;
            const size_t off = ((size_t)h * D + dd) * nq_pad + row0;
            bf16x8 a = *reinterpret_cast<const bf16x8 *>(qt + off);
            bf16x8 b = *reinterpret_cast<const bf16x8 *>(dot + off);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              const bool ok = row0 + i >= lo && row0 + i < hi;
              a[i] = ok ? a[i] : bf16(0.f);
              b[i] = ok ? b[i] : bf16(0.f);
            }
            *reinterpret_cast<bf16x8 *>(Qts + dd * S::TP + 8 * c8) = a;
            *reinterpret_cast<bf16x8 *>(dOts + dd * S::TP + 8 * c8) = b;
          }
          if (tid < kRows) {
            const int64_t row = m * kRows + tid;
            const bool ok = row >= lo && row < hi;
            lse2s[tid] = ok ? lse[(size_t)h * n_q + row] * kLog2e : 0.f;
            dvs[tid] = ok ? dvec[(size_t)h * n_q + row] : 0.f;
          }
          __syncthreads();

          // ---- S = Q K^T and dP = dO V^T, queries on M (lane = key)
          f32x16 sa, pa;
#pragma unroll
          for (int r = 0; r < 16; ++r) { sa[r] = 0.f; pa[r] = 0.f; }
          {
            const bf16 *qp = Qs + perm32(ln) * S::QP + 8 * kg;
            const bf16 *op = dOs + perm32(ln) * S::QP + 8 * kg;
#pragma unroll
            for (int c = 0; c < D / 16; ++c) {
              sa = mfma32(*reinterpret_cast<const bf16x8 *>(qp + 16 * c), kf[c], sa);
              pa = mfma32(*reinterpret_cast<const bf16x8 *>(op + 16 * c), vf[c], pa);
            }
          }
          bf16x8 pb16[2], db16[2];
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int iq = 16 * (r >> 3) + 8 * kg + (r & 7);
            const int64_t row = m * kRows + iq;
            const int64_t qloc = qla + (row - fra);
            const bool ok = key_ok && row >= lo && row < hi && kl <= qloc;
            const float p = ok ? fast_exp2(sa[r] * c2 - lse2s[iq]) : 0.f;
            const float ds = ok ? p * (pa[r] - dvs[iq]) : 0.f;
            pb16[r >> 3][r & 7] = static_cast<bf16>(p);
            db16[r >> 3][r & 7] = static_cast<bf16>(ds);
            Ss[iq * S::SP + 32 * w + ln] = static_cast<bf16>(ds);
          }
          // ---- dV^T += dO^T P, dK^T += Q^T dS (d on M, keys on N, queries on K)
#pragma unroll
          for (int dt = 0; dt < D / 32; ++dt) {
            const bf16 *ap = dOts + (32 * dt + perm32(ln)) * S::TP + 8 * kg;
            const bf16 *bp = Qts + (32 * dt + perm32(ln)) * S::TP + 8 * kg;
#pragma unroll
            for (int c = 0; c < 2; ++c) {
              dva[dt] = mfma32(*reinterpret_cast<const bf16x8 *>(ap + 16 * c), pb16[c], dva[dt]);
              dka[dt] = mfma32(*reinterpret_cast<const bf16x8 *>(bp + 16 * c), db16[c], dka[dt]);
            }
          }
          __syncthreads();
          // ---- dQ = dS K over the 128 keys of the block
          f32x16 qa;
#pragma unroll
          for (int r = 0; r < 16; ++r) qa[r] = 0.f;
          {
            const bf16 *sp = Ss + perm32(ln) * S::SP + 8 * kg;
#pragma unroll
            for (int c = 0; c < S::DQ_CHUNKS; ++c)
              qa = mfma32(*reinterpret_cast<const bf16x8 *>(sp + 16 * (dq_c0 + c)), kq[c], qa);
          }
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int iq = 16 * (r >> 3) + 8 * kg + (r & 7);
            const int64_t row = m * kRows + iq;
            if (row >= lo && row < hi)
              unsafeAtomicAdd(dqacc + ((size_t)row * h_q + h) * D + 32 * dq_dt + ln,
                              qa[r] * scale);
          }
          __syncthreads();
        }
      }
    }

    // ---- write dK, dV for this wave's 32 keys
    if (key_ok) {
      const size_t base = ((size_t)krow * h_kv + g) * D + 8 * kg;
#pragma unroll
      for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
        for (int hh = 0; hh < 2; ++hh) {
          const size_t off = base + 32 * dt + 16 * hh;
          if (accumulate) {
            float *dkp = static_cast<float *>(dk_out) + off;
            float *dvp = static_cast<float *>(dv_out) + off;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              dkp[i] += dka[dt][8 * hh + i] * scale;
              dvp[i] += dva[dt][8 * hh + i];
            }
          } else {
            bf16x8 a, b;
#pragma unroll
            for (int i = 0; i < 8; ++i) {
              a[i] = static_cast<bf16>(dka[dt][8 * hh + i] * scale);
              b[i] = static_cast<bf16>(dva[dt][8 * hh + i]);
            }
            *reinterpret_cast<bf16x8 *>(static_cast<bf16 *>(dk_out) + off) = a;
            *reinterpret_cast<bf16x8 *>(static_cast<bf16 *>(dv_out) + off) = b;
          }
        }
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
static size_t align256b(size_t x) { return (x + 255) / 256 * 256; }

BwdLayout bwd_layout(int64_t T, int64_t n, int64_t n_q, int64_t n_kv, int h_q, int h_kv, int d) {
  (void)T;
  BwdLayout L;
  L.max_items = (n_kv / kBwdBK + n + 1) * (int64_t)h_kv;
  L.nq_pad = (n_q + kRows - 1) / kRows * kRows;
  L.hdr = 0;
  L.ext = align256b(kHdrSlots * sizeof(int32_t));
  L.gmask = align256b(L.ext + (size_t)n * sizeof(int32_t));
  L.items = align256b(L.gmask + (size_t)n * sizeof(unsigned long long));
  L.dvec = align256b(L.items + (size_t)L.max_items * sizeof(BwdItem));
  L.qt = align256b(L.dvec + (size_t)h_q * n_q * sizeof(float));
  L.dot = align256b(L.qt + (size_t)h_q * d * L.nq_pad * sizeof(bf16));
  L.dqacc = align256b(L.dot + (size_t)h_q * d * L.nq_pad * sizeof(bf16));
  L.total = align256b(L.dqacc + (size_t)n_q * h_q * d * sizeof(float));
  return L;
}

template <int D>
static int launch_bwd_d(const bf16 *q, const bf16 *k, const bf16 *v, const bf16 *o,
                        const float *lse, const bf16 *dout, const int64_t *cu, int64_t n,
                        const libra_tile_t *tiles, int64_t T, int64_t n_q, int64_t n_kv, int h_q,
                        int h_kv, float scale, bf16 *dq, void *dk, void *dv, bool accumulate,
                        char *ws, const BwdLayout &L, hipStream_t st, const KernelTimer *tm) {
  int32_t *hdr = reinterpret_cast<int32_t *>(ws + L.hdr);
  int32_t *ext = reinterpret_cast<int32_t *>(ws + L.ext);
  auto *gmask = reinterpret_cast<unsigned long long *>(ws + L.gmask);
  BwdItem *items = reinterpret_cast<BwdItem *>(ws + L.items);
  float *dvec = reinterpret_cast<float *>(ws + L.dvec);
  bf16 *qt = reinterpret_cast<bf16 *>(ws + L.qt);
  bf16 *dot = reinterpret_cast<bf16 *>(ws + L.dot);
  float *dqacc = reinterpret_cast<float *>(ws + L.dqacc);
  static bool attr_set = false;
  if (!attr_set) {
    if (hipFuncSetAttribute(reinterpret_cast<const void *>(&attn_bwd_kernel<D>),
                            hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)BwdShape<D>::SMEM) != hipSuccess)
      return fail(LIBRA_EHIP, "hipFuncSetAttribute failed");
    attr_set = true;
  }
  if (!accumulate) {
    const int64_t n16 = n_kv * h_kv * D * (int64_t)sizeof(bf16) / 16;
    const unsigned blocks = (unsigned)std::min<int64_t>((n16 + 255) / 256, 4096);
    hipLaunchKernelGGL(zero_kernel, dim3(blocks), dim3(256), 0, st, static_cast<uint4 *>(dk), n16);
    hipLaunchKernelGGL(zero_kernel, dim3(blocks), dim3(256), 0, st, static_cast<uint4 *>(dv), n16);
  }
  if (T > 0) {
    hipLaunchKernelGGL(prep_bwd_kernel, dim3(1), dim3(kPrepThreads), 0, st, cu, n, tiles, T, h_q,
                       h_kv, n_q, n_kv, hdr, ext, gmask, items, L.max_items);
    hipLaunchKernelGGL(bwd_pre_kernel<D>, dim3((unsigned)(T * kTileSplit)), dim3(256), 0, st, q, o,
                       dout, tiles, h_q, n_q, n_kv, L.nq_pad, dvec, qt, dot, dqacc);
    int dev = 0, cus = 256;
    hipGetDevice(&dev);
    hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (tm) hipEventRecord(tm->begin, st);
    hipLaunchKernelGGL(attn_bwd_kernel<D>, dim3(cus), dim3(kThreads), BwdShape<D>::SMEM, st, k, v,
                       q, dout, qt, dot, lse, dvec, cu, tiles, T, items, hdr, h_q, h_kv, n_q, n_kv,
                       L.nq_pad, scale, scale * kLog2e, dqacc, dk, dv, accumulate ? 1 : 0);
    if (tm) hipEventRecord(tm->end, st);
    hipLaunchKernelGGL(bwd_finalize_kernel<D>, dim3((unsigned)(T * kTileSplit)), dim3(256), 0, st,
                       tiles, h_q, n_q, n_kv, dqacc, dq);
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(LIBRA_EHIP, "backward launch failed: %s", hipGetErrorString(e));
  return LIBRA_OK;
}

int launch_bwd(const void *q, const void *k, const void *v, const void *o, const float *lse,
               const void *dout, const int64_t *cu, int64_t n, const libra_tile_t *tiles,
               int64_t T, int64_t n_q, int64_t n_kv, int h_q, int h_kv, int d, float scale,
               void *dq, void *dk, void *dv, bool accumulate, void *ws, const BwdLayout &L,
               hipStream_t st, const KernelTimer *tm) {
  auto Q = static_cast<const bf16 *>(q);
  auto K = static_cast<const bf16 *>(k);
  auto V = static_cast<const bf16 *>(v);
  auto O = static_cast<const bf16 *>(o);
  auto dO = static_cast<const bf16 *>(dout);
  auto dQ = static_cast<bf16 *>(dq);
  char *W = static_cast<char *>(ws);
  if (d == 128)
    return launch_bwd_d<128>(Q, K, V, O, lse, dO, cu, n, tiles, T, n_q, n_kv, h_q, h_kv, scale,
                             dQ, dk, dv, accumulate, W, L, st, tm);
  return launch_bwd_d<64>(Q, K, V, O, lse, dO, cu, n, tiles, T, n_q, n_kv, h_q, h_kv, scale, dQ,
                          dk, dv, accumulate, W, L, st, tm);
}

}  // namespace libra
