// dQ kernel of the backward pass (gfx950): query-stationary; its work items
// are the forward's.  Per 64-key block it recomputes S^T = K Q^T and
// dP^T - D = [V | 1] [dO | -D]^T (lane = query; D enters as one extra
// k-block, as in the dK / dV kernel), forms dS^T = P^T * (dP^T - D) on the
// VALU and accumulates dQ^T += K^T dS^T, with the key blocks staged in a
// 4-deep LDS ring.  Two waves share each (head, 32 rows) slice, one per
// 32-key half of every block (see the kernel).
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
  static constexpr int NW = 2 * kWaves;       // waves of the workgroup
  static constexpr int NK = kFwdBN * KC / 64 / NW;   // wave loads per K (V) tile
  static constexpr size_t SMEM = NSTAGE * STAGE * sizeof(bf16);
  // the item-end exchange of the second waves' dQ^T and dS sums fits the ring
  static_assert(kWaves * 64 * (D / 2 + 1) * sizeof(float) <= SMEM, "exchange fits the ring");
};

// Eight waves, two per (query head, 32 rows) slice of the work item: wave
// w + 4 h of slice w takes keys 32 h .. 32 h + 31 of every 64-key block.  Per
// block each wave computes S^T and dP^T - D of its 32 keys, dS^T on the VALU
// (interleaved with its own products) and dQ^T += K^T dS^T, the last one block
// behind, with its dS^T straight from registers (the S^T rows are ordered so
// that its accumulators are the B operand of the dQ^T products).  The two
// halves of a slice add up their dQ^T and sums of dS at the end of the item.
// One barrier per block; a 4-stage K / V ring (block i read by the S^T and
// dP^T products, block i - 1 by the dQ^T products, blocks i + 1 and i + 2
// land).
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
  __shared__ int32_t s_item;
  const int tid = threadIdx.x, l = tid & 63, ln = l & 31, kg = l >> 5;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave index (uniform)
  const int w = wv & (kWaves - 1);                         // slice of the item
  const int hf = wv / kWaves;                              // 32-key half of each block
  int q_serve = blockIdx.x % kXcds, q_left = kXcds;
  const float s_ov = fp16_scale((uint32_t)hdr[kMaxAbs + 1], true) *
                     fp16_scale((uint32_t)hdr[kMaxAbs + 3], true);
  // staging: wave load u covers rows (wv + 8u) * 64 / KC + l / KC of a tile
  auto kst = [&](int u) { return (wv + S::NW * u) * (64 / S::KC) + l / S::KC; };
  uint32_t k_lane[S::NK];
  static_for<S::NK>([&](auto u) {
    const int r = kst(u);
    k_lane[u] = 2u * (uint32_t)(r * h_kv * D + 8 * swt<S::KC>(r, l % S::KC));
  });
  const int prow = perm32(ln) + 32 * hf;
  int koff[D / 16];
  static_for<D / 16>([&](auto c) { koff[c] = prow * D + 8 * swt<S::KC>(prow, 2 * c + kg); });
  // transpose reads of the K^T operands (key chunk 2 hf + c of the block)
  int troff[D / 32][2];
  {
    const int grp = l >> 4, i = (l & 15) >> 2, r = l & 3;
    static_for<D / 32>([&](auto dt) {
      static_for<2>([&](auto h2) {
        const int row = 8 * (grp >> 1) + 4 * h2 + i;
        const int chunk = 4 * dt + 2 * (grp & 1) + (r & 1);
        troff[dt][h2] = row * D + 8 * swt<S::KC>(row, chunk) + 4 * (r >> 1);
      });
    });
  }
  bf16x8 ones3;
  static_for<8>([&](auto i) { ones3[int(i)] = bf16(kg == 0 && i < 3 ? 1.f : 0.f); });

  for (;;) {
    if (tid == 0) s_item = take_item(hdr, kFwdQ, q_serve, q_left);
    __syncthreads();
    const int idx = __builtin_amdgcn_readfirstlane(s_item);
    if (idx < 0) break;
    const FwdItem it = items[idx];
    const int key0 = (int)cu[it.sample];   // n_kv < 2^31 (checked at the boundary)
    const int head = it.head0 + (w % it.nh);
    const int wrow0 = (w / it.nh) * kRows;
    const int wrows = min(max(it.nrows - wrow0, 0), kRows);
    const bool active = wrows > 0;
    const int my_r = active ? min(ln, wrows - 1) : 0;
    const int row = it.q_row0 + wrow0 + my_r;   // Q rows are indexed in 32 bits (FwdItem)
    const int qloc = it.q_loc0 + wrow0 + my_r;
    const int wave_qmin = it.q_loc0 + wrow0;
    const int kb0 = it.kb0, nkb = it.kb1;   // key blocks [kb0, nkb)
    const int wave_nkb = active ? (it.q_loc0 + wrow0 + wrows - 1) / kFwdBN + 1 : 0;
    const int pend = min(wave_nkb, nkb);    // this wave's blocks [kb0, pend)

    // global -> LDS, asynchronous: K and V rows of key block b (keys past the
    // buffer read the last key instead; they are masked)
    auto issue = [&](int b) {
      bf16 *Ks = smem + (b % S::NSTAGE) * S::STAGE;
      bf16 *Vs = Ks + S::K_EL;
      const int kbase = key0 + b * kFwdBN;
      if (kbase + kFwdBN <= n_kv) {
        const size_t off = ((size_t)kbase * h_kv + it.g) * D;
        const uint32_t lk = lds_addr(Ks) + 1024u * wv, lv = lds_addr(Vs) + 1024u * wv;
        if constexpr (S::NK == 2)
          g2l16x4(k + off, v + off, k_lane[0], k_lane[1], lk, lk + S::NW * 1024u, lv,
                  lv + S::NW * 1024u);
        else
          g2l16x2(k + off, v + off, k_lane[0], lk, lv);
        return;
      }
      static_for<S::NK>([&](auto u) {
        const int wl = wv + S::NW * u;
        const int r = kst(u);
        int64_t key = key0 + (int64_t)b * kFwdBN + r;
        key = key < n_kv ? key : n_kv - 1;
        const size_t off = ((size_t)key * h_kv + it.g) * D + 8 * swt<S::KC>(r, l % S::KC);
        g2l16(k + off, Ks + wl * 512);
        g2l16(v + off, Vs + wl * 512);
      });
    };

    // Q and dO rows of this lane's query (B operands), LSE log2(e), and -D
    // (pre-pass value) for dP^T's augmented k-block
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
    if (kb0 < nkb) issue(kb0);
    if (kb0 + 1 < nkb) issue(kb0 + 1);

    f32x16 acc[D / 32];
    static_for<D / 32>([&](auto dt) { acc[dt] = mfma_zero(); });
    bf16x8 dsf[2];          // dS^T of the previous block (B operands, two 16-key chunks)
    float d_run = 0.f;      // this lane's sum of dS over its keys
    // Block b: S^T (8 products at d = 128), the copies of block b + 2 (COPY),
    // dP^T - D (9 products, with the exponentials of P^T on the VALU), then
    // dQ^T += K^T dS^T of block b - 1 (PREV, 8 products) with dS^T of block b
    // on the VALU.  The copies wait behind the other waves' in the memory
    // path; posted here, the S^T products of the wave are already queued on
    // the matrix cores.
    auto block = [&](auto prev_t, auto mask_t, int b, bool copy) {
      constexpr bool PREV = decltype(prev_t)::value, MASK = decltype(mask_t)::value;
      constexpr int NC = D / 16, AHEAD = 3;
      const bf16 *Ks = smem + (b % S::NSTAGE) * S::STAGE, *Vs = Ks + S::K_EL;
      f32x16 sa, pa;
      bf16x8 op[2 * NC];   // MFMA i < NC: S^T from K; NC + c: dP^T from V
      auto rd = [&](auto i) {
        constexpr int kind = i / NC, c = i % NC;
        op[i] = *reinterpret_cast<const bf16x8 *>((kind ? Vs : Ks) + koff[c]);
      };
      static_for<AHEAD>([&](auto i) { rd(i); });
      __builtin_amdgcn_sched_barrier(0);
      static_for<2 * NC>([&](auto i) {
        constexpr int kind = i / NC, c = i % NC;
        if constexpr (kind == 0)
          sa = mfma32(op[i], qf[c], c == 0 ? mfma_zero_c() : sa);
        else
          pa = mfma32(op[i], of[c], c == 0 ? mfma32(ones3, dneg, mfma_zero_c()) : pa);
        if constexpr (i + AHEAD < 2 * NC) rd(std::integral_constant<int, i + AHEAD>{});
        if constexpr (i == NC - 1)
          if (copy) issue(b + 2);
        if constexpr (kind == 1) {
          // P^T = exp2(S^T c2 - LSE log2 e), 16 / NC elements per product
          static_for<16 / NC>([&](auto e) {
            constexpr int r = (16 / NC) * c + e;
            float x = __builtin_fmaf(sa[r], c2, neg_l2);
            if constexpr (MASK) {
              const int kl = b * kFwdBN + 32 * hf + 16 * (r >> 3) + 8 * kg + (r & 7);
              x = kl > qloc ? -INFINITY : x;
            }
            sa[r] = fast_exp2(x);   // P^T in place
          });
        }
        __builtin_amdgcn_sched_barrier(0);
      });
      // dS^T = P^T * (dP^T - D) of block b, under the dQ^T products of block b - 1
      bf16x8 dn[2];
      float dsum = 0.f;
      auto ds_elem = [&](auto rc) {
        constexpr int r = decltype(rc)::value;
        const float ds = sa[r] * pa[r];
        dsum += ds;
        dn[r >> 3][r & 7] = static_cast<bf16>(ds);
      };
      if constexpr (PREV) {
        const bf16 *Kp = smem + ((b - 1) % S::NSTAGE) * S::STAGE + 32 * hf * D;
        constexpr int NT = D / 32, NQ = 2 * NT, TA = 3;   // MFMA j = NT c + dt
        bf16x8 tp[NQ];
        auto rt = [&](auto j) {
          const bf16 *base = Kp + 16 * (j / NT) * D;
          tp[j] = lds_tr16x2(base + troff[j % NT][0], base + troff[j % NT][1]);
        };
        static_for<TA>([&](auto j) { rt(j); });
        static_for<NQ>([&](auto j) {
          acc[j % NT] = mfma32(tp[j], dsf[j / NT], acc[j % NT]);
          if constexpr (j + TA < NQ) rt(std::integral_constant<int, j + TA>{});
          static_for<16 / NQ>([&](auto e) {
            ds_elem(std::integral_constant<int, (16 / NQ) * j + e>{});
          });
          __builtin_amdgcn_sched_barrier(0);
        });
      } else {
        static_for<16>([&](auto r) { ds_elem(r); });
      }
      dsf[0] = dn[0];
      dsf[1] = dn[1];
      return dsum;
    };
    // dQ^T += K^T dS^T of the wave's last block
    auto flush = [&](int b) {
      const bf16 *Kp = smem + (b % S::NSTAGE) * S::STAGE + 32 * hf * D;
      static_for<2 * (D / 32)>([&](auto j) {
        const bf16 *base = Kp + 16 * (j & 1) * D;
        acc[j >> 1] = mfma32(lds_tr16x2(base + troff[j >> 1][0], base + troff[j >> 1][1]),
                             dsf[j & 1], acc[j >> 1]);
      });
    };
    using T_ = std::true_type;
    using F_ = std::false_type;
    // blocks from (wave_qmin + 1) / 64 on reach past the wave's first row
    const int unmasked_end = (wave_qmin + 1) / kFwdBN;
    // iteration i: this wave's copies of block i (block i + 1's may stay in
    // flight), the barrier, then the copies of block i + 2: here for a wave
    // without a block in this iteration, else inside block() (returns true)
    auto step = [&](int i) {
      if (i + 1 < nkb) wait_vm_n<2 * S::NK>();
      else wait_vm();
      barrier_nofence();
      const bool copy = i + 2 < nkb, in_block = copy && i < pend;
      if (copy && !in_block) issue(i + 2);
      return in_block;
    };
    // the first block, the unmasked ones, then the masked ones and the last
    // dQ^T products: one iteration per i in [kb0, nkb] for every wave
    int i = kb0;
    bool cp = step(i);
    if (i < pend)
      d_run += i < unmasked_end ? block(F_{}, F_{}, i, cp) : block(F_{}, T_{}, i, cp);
    const int pipe_end = min(pend, unmasked_end);
    for (++i; i < pipe_end; ++i) {
      cp = step(i);
      d_run += block(T_{}, F_{}, i, cp);
    }
    for (; i <= nkb; ++i) {
      cp = step(i);
      if (i < pend)
        d_run += block(T_{}, T_{}, i, cp);
      else if (i == pend && pend > kb0)
        flush(i - 1);
    }

    // the second half of each slice hands its dQ^T and sum of dS to the first
    // through the ring (every wave is past its last LDS read of the ring)
    float d_half = row_sum2(d_run);
    __syncthreads();
    float *ex = reinterpret_cast<float *>(smem) + (size_t)w * 64 * (D / 2 + 1);
    if (hf == 1) {
      static_for<D / 32>([&](auto dt) {
        static_for<16>([&](auto r) { ex[(dt * 16 + r) * 64 + l] = acc[dt][int(r)]; });
      });
      ex[(D / 2) * 64 + l] = d_half;
    }
    __syncthreads();
    if (hf == 0) {
      static_for<D / 32>([&](auto dt) {
        static_for<16>([&](auto r) { acc[dt][int(r)] += ex[(dt * 16 + r) * 64 + l]; });
      });
      d_half += ex[(D / 2) * 64 + l];
      const float d_exact = dd_q + d_half;
      if (it.slot >= 0) {
        // a part of a split item: unscaled fp32 dQ and its sum of dS, merged by
        // bwd_dq_combine_kernel
        if (active && ln < wrows) {
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
          if (kg == 0)
            parts[(size_t)it.slot * fwd_part_floats(D) + (size_t)kFwdPartRows * D + w * kRows +
                  ln] = d_half;
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
        // D_exact = D + sum_k dS_k (sum_k P_k = 1): the -D record of the dK / dV
        // kernel's augmented operands for this (row, head)
        if (kg == 0) {
          f16x8 rec;
          split3h(-d_exact * s_ov, rec);
          *reinterpret_cast<f16x8 *>(aug + ((size_t)head * (nq_pad / kRows) + row / kRows) *
                                               kAugEl +
                                     kAugEl / 2 + 8 * perm32((int)(row % kRows))) = rec;
        }
      }
    }
    __syncthreads();   // the ring is reused by the next item
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
