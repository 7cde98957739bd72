// dQ kernel of the backward pass (gfx950): query-stationary; its work items
// are the forward's.  Per 64-key block it recomputes S^T = K Q^T and
// dP^T - D = [V | 1] [dO | -D]^T (lane = query; D enters as one extra
// k-block, as in the dK / dV kernel), forms dS^T = P^T * (dP^T - D) on the
// VALU and accumulates dQ^T += K^T dS^T, with the key blocks staged in a
// 4-deep LDS ring.  Producer and consumer waves split this work (see the
// kernel).
//
// It runs before the dK / dV kernel and hands it D: D = rowsum(dO * O) equals
// sum_k P_k dP_k (O = sum_k P_k V_k), which this kernel has in fp32 for every
// key of the row, while the pre-pass can only form it from the bf16-rounded
// O.  Since sum_k P_k = 1, sum_k dS_k = D_exact - D: the row sums of dS (per
// key block, then over blocks) correct the pre-pass value, and replace the -D
// record of the row in the dK / dV kernel's augmented operands; this kernel's
// own dS uses the pre-pass value.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "attn_common.h"
#include "errors.h"

namespace libra {

template <int D>
struct DqShape {
  static constexpr int KC = D / 8;            // 16-byte columns of a K / V row
  static constexpr int K_EL = kFwdBN * D;
  static constexpr int STAGE = 2 * K_EL;      // K and V rows of one key block
  static constexpr int NSTAGE = 4;            // LDS ring of key blocks
  static constexpr int DS_EL = 4 * 64 * 8;    // dS^T of one slice and block (4 KiB)
  static constexpr int NSLOT = 2;             // dS^T hand-over slots per slice
  static constexpr int NK = kFwdBN * KC / 64 / kWaves;   // wave loads per K (V) tile
  // at d = 128 the dynamic LDS is exactly the 160 KiB of a CU
  static constexpr size_t SMEM = (NSTAGE * STAGE + kWaves * NSLOT * DS_EL) * sizeof(bf16);
};

// Eight waves, two per SIMD, in pairs that share a (query head, 32 rows)
// slice of the work item: the producer (waves 0..3) computes S^T and
// dP^T - D on the matrix cores and dS^T on the VALU and hands dS^T over
// through LDS; the consumer (waves 4..7, on the producer's SIMD) stages the
// K / V blocks and accumulates dQ^T += K^T dS^T one block behind.  While one
// wave of a SIMD is on the VALU, the other keeps the matrix cores busy, and
// the copies no longer stall the wave that does the VALU work.  One barrier
// per block; the K / V ring has four stages (producers read block i while
// consumers read block i - 1, and blocks i + 1 and i + 2 land).
template <int D>
__global__ __launch_bounds__(2 * kThreads, 1) void attn_bwd_dq_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ dout, const bf16 *__restrict__ k,
    const bf16 *__restrict__ v, const float *__restrict__ stats,
    const int64_t *__restrict__ cu, const FwdItem *__restrict__ items,
    int32_t *__restrict__ hdr, int h_q, int h_kv, int64_t n_q, int64_t n_kv, int64_t nq_pad,
    float c2, float scale, bf16 *__restrict__ dq, f16 *__restrict__ aug,
    float *__restrict__ parts) {
  using S = DqShape<D>;
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  // the item index lives in the first dS^T slot, free between items
  int32_t &s_item = *reinterpret_cast<int32_t *>(smem + S::NSTAGE * S::STAGE);
  const int tid = threadIdx.x, l = tid & 63, ln = l & 31, kg = l >> 5;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index (uniform)
  const bool producer = wv < kWaves;
  const int w = wv & (kWaves - 1);                         // slice of the item
  // the XCD under round-robin dispatch (the value xcd_of_workgroup() reads;
  // this form gives this kernel the faster schedule)
  int q_serve = blockIdx.x % kXcds, q_left = kXcds;
  bf16 *ds_slots = smem + S::NSTAGE * S::STAGE + w * S::NSLOT * S::DS_EL;
  // scale of -D in the dK / dV kernel's fp16 operands (s_o * s_v, fp16_scale)
  const float s_ov = fp16_scale((uint32_t)hdr[kMaxAbs + 1], true) *
                     fp16_scale((uint32_t)hdr[kMaxAbs + 3], true);
  // staging (consumers): wave load u covers rows (w + 4u) * 64 / KC + l / KC
  // of a tile
  static_assert(S::NK % 2 == 0, "staging copies go four at a time");
  auto kst = [&](int u) { return (w + kWaves * u) * (64 / S::KC) + l / S::KC; };
  const int prow = perm32(ln);
  // A operand of the augmented k-block of dP^T: ones in k = 0, 1, 2
  bf16x8 ones3;
  static_for<8>([&](auto i) { ones3[int(i)] = bf16(kg == 0 && i < 3 ? 1.f : 0.f); });

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

    // global -> LDS (consumers), asynchronous: K and V rows of key block b
    // (keys past the buffer read the last key instead; they are masked);
    // k_lane[u] is the lane's byte offset from the block's first row
    auto issue = [&](int b, const uint32_t (&k_lane)[S::NK]) {
      bf16 *Ks = smem + (b % S::NSTAGE) * S::STAGE;
      bf16 *Vs = Ks + S::K_EL;
      const int64_t kbase = key0 + (int64_t)b * kFwdBN;
      if (kbase + kFwdBN <= n_kv) {
        const size_t off = ((size_t)kbase * h_kv + it.g) * D;
        const uint32_t lk = lds_addr(Ks) + 1024u * w, lv = lds_addr(Vs) + 1024u * w;
        static_for<S::NK / 2>([&](auto h) {
          constexpr uint32_t d0 = 2 * h * kWaves * 1024u, d1 = d0 + kWaves * 1024u;
          g2l16x4(k + off, v + off, k_lane[2 * h], k_lane[2 * h + 1], lk + d0, lk + d1, lv + d0,
                  lv + d1);
        });
        return;
      }
      static_for<S::NK>([&](auto u) {
        const int wl = w + kWaves * u;
        const int r = kst(u);
        int64_t key = key0 + (int64_t)b * kFwdBN + r;
        key = key < n_kv ? key : n_kv - 1;
        const size_t off = ((size_t)key * h_kv + it.g) * D + 8 * swt<S::KC>(r, l % S::KC);
        g2l16(k + off, Ks + wl * 512);
        g2l16(v + off, Vs + wl * 512);
      });
    };

    if (producer) {
      // per-lane LDS offsets (elements) of the K / V rows perm32(ln) for S^T and dP^T
      int koff[D / 16];
      static_for<D / 16>([&](auto c) { koff[c] = prow * D + 8 * swt<S::KC>(prow, 2 * c + kg); });
      // ---- producer: Q and dO rows of this lane's query (B operands),
      // LSE log2(e), and -D (pre-pass value) for dP^T's augmented k-block
      bf16x8 qf[D / 16], of[D / 16], dneg;
      float l2 = 0.f, dd_q = 0.f;
      if (active) {
        const size_t off = ((size_t)row * h_q + head) * D + 8 * kg;
#pragma unroll
        for (int c = 0; c < D / 16; ++c) {
          qf[c] = *reinterpret_cast<const bf16x8 *>(q + off + 16 * c);
          of[c] = *reinterpret_cast<const bf16x8 *>(dout + off + 16 * c);
        }
        const float *st = stats + ((size_t)head * (nq_pad / kRows) + row / kRows) * 2 * kRows;
        l2 = st[row % kRows];
        dd_q = st[kRows + row % kRows];
      }
      split3(kg == 0 ? -dd_q : 0.f, dneg);
      const float neg_l2 = -l2;
      wait_vm_known();
      // S^T and dP^T - D of block b (keys on M, queries on N), then
      // dS^T = P^T * (dP^T - D), P^T = exp2(S^T c2 - LSE log2 e) (with MASK,
      // keys after the lane's query give P = 0), into hand-over slot `slot`.
      // Returns this lane's sum of dS over the block.
      auto block = [&](auto mask_t, int b, bf16 *slot) {
        constexpr bool MASK = decltype(mask_t)::value;
        constexpr int NC = D / 16, NM = 4 * NC, AHEAD = 4;
        const bf16 *Ks = smem + (b % S::NSTAGE) * S::STAGE, *Vs = Ks + S::K_EL;
        f32x16 sa[2], pa[2];
        // MFMA i = 2 NC t + 2 c + kind (kind 0: S^T from K, 1: dP^T from V);
        // each operand is read AHEAD MFMAs before its product
        bf16x8 op[NM];
        auto rd = [&](auto i) {
          constexpr int t = i / (2 * NC), c = (i % (2 * NC)) / 2, kind = i % 2;
          op[i] = *reinterpret_cast<const bf16x8 *>((kind ? Vs : Ks) + 32 * t * D + koff[c]);
        };
        bf16x8 dsf[4];
        float dsum = 0.f;
        auto elem = [&](auto t, auto r) {
          float x = __builtin_fmaf(sa[t][int(r)], c2, neg_l2);
          if constexpr (MASK) {
            const int kl = b * kFwdBN + 32 * t + 16 * (r >> 3) + 8 * kg + (r & 7);
            x = kl > qloc ? -INFINITY : x;
          }
          const float ds = fast_exp2(x) * pa[t][int(r)];
          dsum += ds;
          dsf[2 * t + (r >> 3)][r & 7] = static_cast<bf16>(ds);
        };
        static_for<AHEAD>([&](auto i) { rd(i); });
        __builtin_amdgcn_sched_barrier(0);
        // the products of the second 32-key tile carry the VALU work of the
        // first
        constexpr int EPM = 16 / (2 * NC);   // elements of tile 0 per product of tile 1
        static_for<NM>([&](auto i) {
          constexpr int t = i / (2 * NC), c = (i % (2 * NC)) / 2, kind = i % 2;
          if constexpr (kind == 0)
            sa[t] = mfma32(op[i], qf[c], c == 0 ? mfma_zero_c() : sa[t]);
          else
            pa[t] = mfma32(op[i], of[c],
                           c == 0 ? mfma32(ones3, dneg, mfma_zero_c()) : pa[t]);
          if constexpr (i + AHEAD < NM) rd(std::integral_constant<int, i + AHEAD>{});
          if constexpr (t == 1)
            static_for<EPM>([&](auto e) {
              elem(std::integral_constant<int, 0>{},
                   std::integral_constant<int, EPM * (i - 2 * NC) + e>{});
            });
          __builtin_amdgcn_sched_barrier(0);
        });
        static_for<16>([&](auto r) { elem(std::integral_constant<int, 1>{}, r); });
        static_for<4>([&](auto c) {
          *reinterpret_cast<bf16x8 *>(slot + (c * 64 + l) * 8) = dsf[c];
        });
        return dsum;
      };
      float d_run = 0.f;   // this lane's half of sum_k dS_k over the row's keys
      for (int i = kb0; i <= nkb; ++i) {
        // block i landed for every wave; dS^T of block i - 1 is in its slot
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        barrier_nofence();
        // a part of a split item ends at nkb below the wave's last block
        if (i < wave_nkb && i < nkb) {
          bf16 *slot = ds_slots + (i & 1) * S::DS_EL;
          if (i * kFwdBN + kFwdBN - 1 > wave_qmin)   // reaches past the wave's first row
            d_run += block(std::true_type{}, i, slot);
          else
            d_run += block(std::false_type{}, i, slot);
        }
      }
      // D_exact = D + sum_k dS_k (sum_k P_k = 1): the -D record of the dK / dV
      // kernel's augmented operands for this (row, head)
      const float d_part = row_sum2(d_run);
      const float d_exact = dd_q + d_part;
      if (it.slot >= 0) {
        // a part of a split item: its sum of dS, merged by bwd_dq_combine_kernel
        if (active && ln < wrows && kg == 0)
          parts[(size_t)it.slot * fwd_part_floats(D) + (size_t)kFwdPartRows * D + w * kRows + ln] =
              d_part;
      } else if (active && ln < wrows && kg == 0) {
        f16x8 rec;
        split3h(-d_exact * s_ov, rec);
        *reinterpret_cast<f16x8 *>(aug + ((size_t)head * (nq_pad / kRows) + row / kRows) * kAugEl +
                                   kAugEl / 2 + 8 * perm32((int)(row % kRows))) = rec;
      }
    } else {
      // ---- consumer: stages K / V one block ahead, accumulates dQ^T; the
      // per-lane LDS offsets of the transpose reads of the K tile (K^T)
      int troff[D / 32][2];
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
      uint32_t k_lane[S::NK];
      static_for<S::NK>([&](auto u) {
        const int r = kst(u);
        k_lane[u] = 2u * (uint32_t)(r * h_kv * D + 8 * swt<S::KC>(r, l % S::KC));
      });
      f32x16 acc[D / 32];
      static_for<D / 32>([&](auto dt) { acc[dt] = mfma_zero(); });
      if (kb0 < nkb) issue(kb0, k_lane);
      if (kb0 + 1 < nkb) issue(kb0 + 1, k_lane);
      for (int i = kb0; i <= nkb; ++i) {
        // this wave's copies of block i (block i + 1's may stay in flight)
        if (i + 1 < nkb) wait_vm_n<2 * S::NK>();
        else wait_vm();
        barrier_nofence();
        if (i + 2 < nkb) issue(i + 2, k_lane);
        const int b = i - 1;
        if (b >= kb0 && b < wave_nkb) {
          const bf16 *Ks = smem + (b % S::NSTAGE) * S::STAGE;
          const bf16 *slot = ds_slots + (b & 1) * S::DS_EL;
          bf16x8 dsf[4];
          static_for<4>([&](auto c) {
            dsf[c] = *reinterpret_cast<const bf16x8 *>(slot + (c * 64 + l) * 8);
          });
          // MFMA j = 4 dt + c: key chunk c = 16 keys from tile row 16 c;
          // transpose operands read TA MFMAs ahead
          constexpr int NQ = 4 * (D / 32), TA = 3;
          bf16x8 tp[NQ];
          auto rt = [&](auto j) {
            const bf16 *base = Ks + 16 * (j & 3) * D;
            tp[j] = lds_tr16x2(base + troff[j >> 2][0], base + troff[j >> 2][1]);
          };
          static_for<TA>([&](auto j) { rt(j); });
          static_for<NQ>([&](auto j) {
            acc[j >> 2] = mfma32(tp[j], dsf[j & 3], acc[j >> 2]);
            if constexpr (j + TA < NQ) rt(std::integral_constant<int, j + TA>{});
            __builtin_amdgcn_sched_barrier(0);
          });
        }
      }
      if (active && ln < wrows && it.slot >= 0) {
        // a part of a split item: unscaled fp32 dQ into its partial slot
        float *op = parts + (size_t)it.slot * fwd_part_floats(D) + (size_t)(w * kRows + ln) * D +
                    8 * kg;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            float4 *dst = reinterpret_cast<float4 *>(op + 32 * dt + 16 * hh);
            dst[0] = make_float4(acc[dt][8 * hh], acc[dt][8 * hh + 1], acc[dt][8 * hh + 2],
                                 acc[dt][8 * hh + 3]);
            dst[1] = make_float4(acc[dt][8 * hh + 4], acc[dt][8 * hh + 5], acc[dt][8 * hh + 6],
                                 acc[dt][8 * hh + 7]);
          }
      } else if (active && ln < wrows) {
        bf16 *op = dq + ((size_t)row * h_q + head) * D + 8 * kg;
#pragma unroll
        for (int dt = 0; dt < D / 32; ++dt)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            bf16x8 ov;
#pragma unroll
            for (int i = 0; i < 8; ++i) ov[i] = static_cast<bf16>(acc[dt][8 * hh + i] * scale);
            *reinterpret_cast<bf16x8 *>(op + 32 * dt + 16 * hh) = ov;
          }
      }
    }
    __syncthreads();   // the ring and the slots are reused by the next item
  }
}

// Merges the parts of every split item (hdr[kFwdSplits] records): dQ is the
// scaled sum of the parts' fp32 dQ; D_exact = D + the parts' sums of dS gives
// the -D record of the dK / dV kernel, as the dQ kernel writes it for whole
// items.  Two threads per row (half of the head dimension each).
template <int D>
__global__ __launch_bounds__(256) void bwd_dq_combine_kernel(
    const FwdSplit *__restrict__ splits, const int32_t *__restrict__ hdr,
    const float *__restrict__ parts, const float *__restrict__ stats, int h_q, int64_t nq_pad,
    float scale, bf16 *__restrict__ dq, f16 *__restrict__ aug) {
  constexpr size_t PF = fwd_part_floats(D);
  const int count = hdr[kFwdSplits];
  const float s_ov = fp16_scale((uint32_t)hdr[kMaxAbs + 1], true) *
                     fp16_scale((uint32_t)hdr[kMaxAbs + 3], true);
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
    float acc[D / 2];
#pragma unroll
    for (int i = 0; i < D / 2; ++i) acc[i] = 0.f;
    float dsum = 0.f;
    for (int p = 0; p < sp.parts; ++p) {
      const float *rec = parts + (size_t)(sp.base + p) * PF;
      dsum += rec[(size_t)kFwdPartRows * D + pr];
      const float4 *src = reinterpret_cast<const float4 *>(rec + (size_t)pr * D + half * (D / 2));
#pragma unroll
      for (int i = 0; i < D / 8; ++i) {
        const float4 x = src[i];
        acc[4 * i] += x.x;
        acc[4 * i + 1] += x.y;
        acc[4 * i + 2] += x.z;
        acc[4 * i + 3] += x.w;
      }
    }
    bf16 *op = dq + ((size_t)row * h_q + head) * D + half * (D / 2);
#pragma unroll
    for (int i = 0; i < D / 16; ++i) {
      bf16x8 ov;
#pragma unroll
      for (int j = 0; j < 8; ++j) ov[j] = static_cast<bf16>(acc[8 * i + j] * scale);
      *reinterpret_cast<bf16x8 *>(op + 8 * i) = ov;
    }
    if (half == 0) {
      const size_t blk = (size_t)head * (nq_pad / kRows) + row / kRows;
      const float d_exact = stats[blk * 2 * kRows + kRows + row % kRows] + dsum;
      f16x8 rec;
      split3h(-d_exact * s_ov, rec);
      *reinterpret_cast<f16x8 *>(aug + blk * kAugEl + kAugEl / 2 + 8 * perm32((int)(row % kRows))) =
          rec;
    }
  }
}

int launch_bwd_dq(int d, const bf16 *q, const bf16 *dout, const bf16 *k, const bf16 *v,
                  const float *stats, const int64_t *cu, const FwdItem *items, int32_t *hdr,
                  int h_q, int h_kv, int64_t n_q, int64_t n_kv, int64_t nq_pad, float scale,
                  bf16 *dq, f16 *aug, const FwdSplit *splits, float *parts, int max_parts,
                  int blocks, hipStream_t st, const KernelTimer *tm) {
  static bool attr_set[2] = {false, false};
  const int which = d == 128 ? 1 : 0;
  const void *fn = d == 128 ? reinterpret_cast<const void *>(&attn_bwd_dq_kernel<128>)
                            : reinterpret_cast<const void *>(&attn_bwd_dq_kernel<64>);
  const size_t smem = d == 128 ? DqShape<128>::SMEM : DqShape<64>::SMEM;
  if (!attr_set[which]) {
    if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)smem) !=
        hipSuccess)
      return fail(LIBRA_EHIP, "cannot reserve %zu bytes of LDS for the dQ kernel", smem);
    attr_set[which] = true;
  }
  if (tm) hipEventRecord(tm->begin, st);
  if (d == 128) {
    hipLaunchKernelGGL(attn_bwd_dq_kernel<128>, dim3(blocks), dim3(2 * kThreads), smem, st, q, dout,
                       k, v, stats, cu, items, hdr, h_q, h_kv, n_q, n_kv, nq_pad, scale * kLog2e,
                       scale, dq, aug, parts);
    if (max_parts > 0)
      hipLaunchKernelGGL(bwd_dq_combine_kernel<128>, dim3(blocks), dim3(256), 0, st, splits, hdr,
                         parts, stats, h_q, nq_pad, scale, dq, aug);
  } else {
    hipLaunchKernelGGL(attn_bwd_dq_kernel<64>, dim3(blocks), dim3(2 * kThreads), smem, st, q, dout,
                       k, v, stats, cu, items, hdr, h_q, h_kv, n_q, n_kv, nq_pad, scale * kLog2e,
                       scale, dq, aug, parts);
    if (max_parts > 0)
      hipLaunchKernelGGL(bwd_dq_combine_kernel<64>, dim3(blocks), dim3(256), 0, st, splits, hdr,
                         parts, stats, h_q, nq_pad, scale, dq, aug);
  }
  if (tm) hipEventRecord(tm->end, st);
  return LIBRA_OK;
}

}  // namespace libra
