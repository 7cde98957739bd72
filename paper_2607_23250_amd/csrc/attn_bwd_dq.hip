// dQ kernel of the backward pass (gfx950): query-stationary and shaped like the
// forward; its work items are the forward's.  Per 64-key block it recomputes
// S^T = K Q^T and dP^T - D = [V | 1] [dO | -D]^T (lane = query; D enters as
// one extra k-block, as in the dK / dV kernel), forms
// dS^T = P^T * (dP^T - D) on the VALU and accumulates dQ^T += K^T dS^T, with
// the key blocks staged in a 4-deep LDS ring.  The VALU work of one key block
// overlaps the S^T / dP^T products of the next.
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
  static constexpr int STAGE = 2 * K_EL;
  static constexpr int NSTAGE = 4;            // LDS ring of key blocks
  static constexpr int NK = kFwdBN * KC / 64 / kWaves;   // wave loads per K (V) tile
  static constexpr int LOADS = 2 * NK;                    // per wave per block
  static constexpr size_t SMEM = NSTAGE * STAGE * sizeof(bf16);
  static_assert((NSTAGE - 1) * LOADS <= 63, "vmcnt range");
};

template <int D>
__global__ __launch_bounds__(kThreads, 1) void attn_bwd_dq_kernel(
    const bf16 *__restrict__ q, const bf16 *__restrict__ dout, const bf16 *__restrict__ k,
    const bf16 *__restrict__ v, const float *__restrict__ stats,
    const int64_t *__restrict__ cu, const FwdItem *__restrict__ items,
    int32_t *__restrict__ hdr, int h_q, int h_kv, int64_t n_q, int64_t n_kv, int64_t nq_pad,
    float c2, float scale, bf16 *__restrict__ dq, f16 *__restrict__ aug) {
  using S = DqShape<D>;
  extern __shared__ __attribute__((aligned(16))) bf16 smem[];
  __shared__ int32_t s_item;
  const int tid = threadIdx.x, l = tid & 63, ln = l & 31, kg = l >> 5;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index (uniform)
  int q_serve = blockIdx.x % kXcds, q_left = kXcds;
  // scale of -D in the dK / dV kernel's fp16 operands (s_o * s_v, fp16_scale)
  const float s_ov = fp16_scale((uint32_t)hdr[kMaxAbs + 1], true) *
                     fp16_scale((uint32_t)hdr[kMaxAbs + 3], true);
  // per-lane LDS offsets (elements): K / V rows perm32(ln) for S^T and dP^T,
  // and the transpose reads of the K tile that give the K^T operand of dQ^T
  // (as in the dK/dV kernel, with keys in place of query rows)
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
  static_assert(S::NK % 2 == 0, "staging copies go four at a time");
  auto kst = [&](int u) { return (w + kWaves * u) * (64 / S::KC) + l / S::KC; };
  uint32_t k_lane[S::NK];
  static_for<S::NK>([&](auto u) {
    const int r = kst(u);
    k_lane[u] = 2u * (uint32_t)(r * h_kv * D + 8 * swt<S::KC>(r, l % S::KC));
  });
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
    const int nkb = (it.q_loc0 + it.nrows - 1) / kFwdBN + 1;
    const int wave_nkb = active ? (it.q_loc0 + wrow0 + wrows - 1) / kFwdBN + 1 : 0;

    bf16x8 qf[D / 16], of[D / 16];
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
    // -D as the B operand of dP^T's augmented k-block: [V | 1] [dO | -D]^T
    bf16x8 dneg;
    split3(kg == 0 ? -dd_q : 0.f, dneg);

    wait_vm_known();
    f32x16 acc[D / 32];
    static_for<D / 32>([&](auto dt) { acc[dt] = mfma_zero(); });

    // global -> LDS, asynchronous: K and V rows of key block b (keys past the
    // buffer read the last key instead; they are masked)
    auto issue = [&](int b, int sg) {
      bf16 *Ks = smem + sg * S::STAGE;
      bf16 *Vs = Ks + S::K_EL;
      const int64_t kb0 = key0 + (int64_t)b * kFwdBN;
      if (kb0 + kFwdBN <= n_kv) {
        const size_t off = ((size_t)kb0 * h_kv + it.g) * D;
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

    // Key blocks in a ring of NSTAGE one-block stages, block b in stage
    // b % NSTAGE.  Iteration b forms dS^T of block b on the VALU while the
    // MFMAs compute S^T and dP^T of block b + 1 (two register sets, used in
    // turn), then accumulates dQ^T += K^T dS^T of block b.
    auto stage = [&](int b) { return smem + (b & (S::NSTAGE - 1)) * S::STAGE; };
    using Acc2 = f32x16[2];
    // S^T and dP^T of block b (keys on M, queries on N)
    auto sdp = [&](int b, Acc2 &s, Acc2 &dp) {
      const bf16 *Ks = stage(b), *Vs = Ks + S::K_EL;
      static_for<2>([&](auto t) {
        static_for<16>([&](auto r) { s[t][int(r)] = 0.f; });
        dp[t] = mfma32(ones3, dneg, mfma_zero_c());
        static_for<D / 16>([&](auto c) {
          s[t] = mfma32(*reinterpret_cast<const bf16x8 *>(Ks + 32 * t * D + koff[c]), qf[c], s[t]);
          dp[t] = mfma32(*reinterpret_cast<const bf16x8 *>(Vs + 32 * t * D + koff[c]), of[c],
                         dp[t]);
        });
      });
    };
    // One element of dS^T = P^T * (dP^T - D) of the block in (s, dp), the
    // products having subtracted D already:
    // register r of tile t, with P^T = exp2(S^T c2 - LSE log2 e); with MASK,
    // keys after the lane's query give P = 0
    const float neg_l2 = -l2;
    auto ds_elem = [&](auto mask_t, auto t, auto r, int b, Acc2 &s, Acc2 &dp,
                       bf16x8 (&dsf)[4], float &pdp) {
      float x = __builtin_fmaf(s[t][int(r)], c2, neg_l2);
      if constexpr (decltype(mask_t)::value) {
        const int kl = b * kFwdBN + 32 * t + 16 * (r >> 3) + 8 * kg + (r & 7);
        x = kl > qloc ? -INFINITY : x;
      }
      const float ds = fast_exp2(x) * dp[t][int(r)];
      pdp += ds;
      dsf[2 * t + (r >> 3)][r & 7] = static_cast<bf16>(ds);
    };
    // dQ^T += K^T dS^T of block b; key chunk c = 16 keys from tile row 16 c.
    // MFMA i = 4 dt + c; its transpose operand is read three MFMAs ahead.
    auto dqm = [&](int b, const bf16x8 (&dsf)[4]) {
      const bf16 *Ks = stage(b);
      constexpr int NM = 4 * (D / 32), AHEAD = 3;
      bf16x8 op[NM];
      auto rd = [&](auto i) {
        const bf16 *base = Ks + 16 * (i & 3) * D;
        op[i] = lds_tr16x2(base + troff[i >> 2][0], base + troff[i >> 2][1]);
      };
      static_for<AHEAD>([&](auto i) { rd(i); });
      static_for<NM>([&](auto i) {
        acc[i >> 2] = mfma32(op[i], dsf[i & 3], acc[i >> 2]);
        if constexpr (i + AHEAD < NM) rd(std::integral_constant<int, i + AHEAD>{});
        __builtin_amdgcn_sched_barrier(0);
      });
    };
    // phase A: dS^T of block b from (sc, dc) on the VALU, spread evenly over
    // the MFMAs of S^T / dP^T of block b + 1 into (sn, dn) when `next`.  MFMA
    // i = 2 NC t + 2 c + kind (kind 0: S^T from K, 1: dP^T from V); its K / V
    // operand is read four MFMAs ahead.
    auto phase_a = [&](auto mask_t, auto next_t, int b, Acc2 &sc, Acc2 &dc, Acc2 &sn, Acc2 &dn,
                       bf16x8 (&dsf)[4], float &pdp) {
      if constexpr (decltype(next_t)::value) {
        const bf16 *Ks = stage(b + 1), *Vs = Ks + S::K_EL;
        constexpr int NC = D / 16, NM = 4 * NC, AHEAD = 4;
        static_assert(32 % NM == 0, "dS elements spread evenly over the MFMAs");
        constexpr int EPM = 32 / NM;     // dS elements per MFMA
        bf16x8 op[NM];
        auto rd = [&](auto i) {
          constexpr int t = i / (2 * NC), c = (i % (2 * NC)) / 2, kind = i % 2;
          op[i] = *reinterpret_cast<const bf16x8 *>((kind ? Vs : Ks) + 32 * t * D + koff[c]);
        };
        static_for<AHEAD>([&](auto i) { rd(i); });
        __builtin_amdgcn_sched_barrier(0);
        static_for<NM>([&](auto i) {
          constexpr int t = i / (2 * NC), c = (i % (2 * NC)) / 2, kind = i % 2;
          Acc2 &dst = kind ? dn : sn;
          const bf16x8 &bop = kind ? of[c] : qf[c];
          if constexpr (c == 0 && kind == 1)
            dst[t] = mfma32(op[i], bop, mfma32(ones3, dneg, mfma_zero_c()));
          else
            dst[t] = mfma32(op[i], bop, c == 0 ? mfma_zero_c() : dst[t]);
          if constexpr (i + AHEAD < NM) rd(std::integral_constant<int, i + AHEAD>{});
          static_for<EPM>([&](auto e) {
            constexpr int j = EPM * i + e;
            ds_elem(mask_t, std::integral_constant<int, j / 16>{},
                    std::integral_constant<int, j % 16>{}, b, sc, dc, dsf, pdp);
          });
          __builtin_amdgcn_sched_barrier(0);
        });
      } else {
        static_for<2>([&](auto t) {
          static_for<16>([&](auto r) { ds_elem(mask_t, t, r, b, sc, dc, dsf, pdp); });
        });
      }
    };

    int issued = 0;
    for (; issued < nkb && issued < S::NSTAGE - 1; ++issued) issue(issued, issued);
    float d_run = 0.f;   // this lane's half of sum_k dS_k over the row's keys
    auto iter = [&](int b, Acc2 &sc, Acc2 &dc, Acc2 &sn, Acc2 &dn) {
      if (b + 1 < nkb) {
        // block b + 1 landed (at most one later block in flight) and every
        // wave is done with block b - 1, whose stage takes block b + 3
        wait_stages<S::LOADS, 1>(issued - 2 - b);
        barrier_nofence();
        if (issued < nkb) {
          issue(issued, issued & (S::NSTAGE - 1));
          ++issued;
        }
      }
      if (b < wave_nkb) {
        bf16x8 dsf[4];
        float pdp = 0.f;                                         // this block's sum of dS
        const bool mask = b * kFwdBN + kFwdBN - 1 > wave_qmin;   // reaches past the first row
        if (b + 1 < wave_nkb) {
          if (mask) phase_a(std::true_type{}, std::true_type{}, b, sc, dc, sn, dn, dsf, pdp);
          else phase_a(std::false_type{}, std::true_type{}, b, sc, dc, sn, dn, dsf, pdp);
        } else {
          if (mask) phase_a(std::true_type{}, std::false_type{}, b, sc, dc, sn, dn, dsf, pdp);
          else phase_a(std::false_type{}, std::false_type{}, b, sc, dc, sn, dn, dsf, pdp);
        }
        d_run += pdp;
        dqm(b, dsf);
      }
    };
    f32x16 sA[2], dA[2], sB[2], dB[2];
    if (nkb > 0) {
      wait_stages<S::LOADS, S::NSTAGE - 2>(issued - 1);
      barrier_nofence();
      if (wave_nkb > 0) {
        sdp(0, sA, dA);
        sched_pipeline<4 * (D / 16), 4>();
      }
    }
    for (int b = 0; b < nkb; b += 2) {
      iter(b, sA, dA, sB, dB);
      if (b + 1 < nkb) iter(b + 1, sB, dB, sA, dA);
    }
    wait_vm_n<0>();
    __syncthreads();   // the ring is reused by the next item

    // D_exact = D + sum_k dS_k (sum_k P_k = 1)
    const float d_exact = dd_q + row_sum2(d_run);
    if (active && ln < wrows && kg == 0) {
      f16x8 rec;
      split3h(-d_exact * s_ov, rec);
      *reinterpret_cast<f16x8 *>(aug + ((size_t)head * (nq_pad / kRows) + row / kRows) * kAugEl +
                                 kAugEl / 2 + 8 * perm32((int)(row % kRows))) = rec;
    }
    if (active && ln < wrows) {
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
}

int launch_bwd_dq(int d, const bf16 *q, const bf16 *dout, const bf16 *k, const bf16 *v,
                  const float *stats, const int64_t *cu, const FwdItem *items, int32_t *hdr,
                  int h_q, int h_kv, int64_t n_q, int64_t n_kv, int64_t nq_pad, float scale,
                  bf16 *dq, f16 *aug, int blocks, hipStream_t st, const KernelTimer *tm) {
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
  if (d == 128)
    hipLaunchKernelGGL(attn_bwd_dq_kernel<128>, dim3(blocks), dim3(kThreads), smem, st, q, dout,
                       k, v, stats, cu, items, hdr, h_q, h_kv, n_q, n_kv, nq_pad, scale * kLog2e,
                       scale, dq, aug);
  else
    hipLaunchKernelGGL(attn_bwd_dq_kernel<64>, dim3(blocks), dim3(kThreads), smem, st, q, dout,
                       k, v, stats, cu, items, hdr, h_q, h_kv, n_q, n_kv, nq_pad, scale * kLog2e,
                       scale, dq, aug);
  if (tm) hipEventRecord(tm->end, st);
  return LIBRA_OK;
}

}  // namespace libra
