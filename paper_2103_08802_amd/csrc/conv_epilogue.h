// Epilogue of the grouped convolution kernels (forward and data gradient), shared by the
// implicit-GEMM kernels of k_conv.hip and k_gemm.hip.
#pragma once
#include "bn_fuse.h"
#include "device_common.h"
#include "pnn_internal.h"

namespace pnn {

// The epilogue shared by the convolution kernels, once the workgroup's fp32 tile (BM rows x BNc
// columns from n0, row stride LDA) is staged in acc_s: residual / addend, BN-mask and BN-apply
// forms, 16-byte stores, and the per-tile BN partials of the stored result (EPI_BN_FUSE: and the
// statistics finalised from them by the last workgroup, bn_fwd_fuse).  Each thread owns
// 16-byte column chunks of rows tid / ncc + k * rpp; pre / pre2 hold the streamed epilogue operands
// of those chunks (loaded by the caller); piv_s is BNc floats of LDS for the forward pivot; bn is
// [7][BNS] floats of LDS (mean, invstd, scale, shift; A, B, K) for the data-gradient BN forms.
template <typename T, int MODE, int BM, int BNc, int LDA, int BNS>
__device__ __forceinline__ void conv_epilogue(const ConvProb& P, float* acc_s, float* piv_s, const float* bn, int tm,
                                              int n0, const uint4* pre, const uint4* pre2) {
  constexpr int VE = St<T>::VE;
  constexpr int STAT_WORDS = 2 * 256 * VE + 512;
  constexpr int ACC_WORDS = BM * LDA > STAT_WORDS ? BM * LDA : STAT_WORDS;
  constexpr int ncc = BNc / VE;
  constexpr int rpp = 256 / ncc;
  constexpr int NCH = BM / rpp;
  const int tid = threadIdx.x;
  const int c0 = (tid % ncc) * VE;
  const bool bnmask = MODE == MODE_BWD && (P.flags & (EPI_BN_MASK | EPI_BN_APPLY));
  const bool bnapply = MODE == MODE_BWD && (P.flags & EPI_BN_APPLY);
  // Forward BN statistics are summed about a per-tile pivot, the tile's first stored row (kept in
  // piv_s): (sum d, sum d^2) with d = value - pivot do not cancel when a
  // channel's mean is large against its spread; the tile's mean and sum of squared deviations are
  // formed from them below.
  const bool fstats = MODE == MODE_FWD && (P.flags & EPI_STATS) != 0;
  float pv[VE];
  if (fstats) {
    if (tid < ncc) {                   // the threads that hold the tile's first row
      Chunk<T> r0, x0;
      unpack_chunk<T>(pre[0], r0);
      unpack_chunk<T>(pre2[0], x0);
#pragma unroll
      for (int e = 0; e < VE; ++e)
        piv_s[c0 + e] = St<T>::rnd(acc_s[c0 + e] + (P.res ? r0.v[e] : 0.f) + (P.ext ? x0.v[e] : 0.f));
    }
    __syncthreads();
  }
#pragma unroll
  for (int e = 0; e < VE; ++e) pv[e] = fstats ? piv_s[c0 + e] : 0.f;

  float s1[VE], s2[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) s1[e] = s2[e] = 0.f;
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    const int r = tid / ncc + k * rpp;
    const int m = tm * BM + r;
    if (m >= P.M) break;
    Chunk<T> pfc;
    unpack_chunk<T>(pre[k], pfc);
    const long idx = (long)m * P.ncol + n0 + c0;
    float v[VE];
#pragma unroll
    for (int e = 0; e < VE; ++e) v[e] = acc_s[r * LDA + c0 + e];
    if constexpr (MODE == MODE_FWD) {
      if (P.res) {
#pragma unroll
        for (int e = 0; e < VE; ++e) v[e] += pfc.v[e];
      }
      if (P.ext) {
        Chunk<T> x;
        unpack_chunk<T>(pre2[k], x);
#pragma unroll
        for (int e = 0; e < VE; ++e) v[e] += x.v[e];
      }
      store_chunk<T>(P.out, idx, v);
#pragma unroll
      for (int e = 0; e < VE; ++e) {
        const float d = St<T>::rnd(v[e]) - pv[e];
        s1[e] += d;
        s2[e] += d * d;
      }
    } else {
      if (P.flags & EPI_ACC_IN) {
#pragma unroll
        for (int e = 0; e < VE; e += 4) {
          const float4 x = *(const float4*)(P.acc_in + idx + e);
          v[e] += x.x; v[e + 1] += x.y; v[e + 2] += x.z; v[e + 3] += x.w;
        }
      }
      if (P.flags & EPI_STORE_F32) {
#pragma unroll
        for (int e = 0; e < VE; e += 4) *(float4*)(P.out32 + idx + e) = make_float4(v[e], v[e + 1], v[e + 2], v[e + 3]);
      } else if (bnmask) {
        const Chunk<T>& z = pfc;
        float mu[VE], is[VE], sc[VE], sh[VE];
#pragma unroll
        for (int e = 0; e < VE; e += 4) {
          *(float4*)&mu[e] = *(const float4*)&bn[0 * BNS + c0 + e];
          *(float4*)&is[e] = *(const float4*)&bn[1 * BNS + c0 + e];
          *(float4*)&sc[e] = *(const float4*)&bn[2 * BNS + c0 + e];
          *(float4*)&sh[e] = *(const float4*)&bn[3 * BNS + c0 + e];
        }
#pragma unroll
        for (int e = 0; e < VE; ++e) v[e] = fmaf(z.v[e], sc[e], sh[e]) > 0.f ? v[e] : 0.f;
        if (bnapply) {
          // the BN backward apply of the stored-dbn path, on dbn rounded as it would be stored
          float ca[VE], cb[VE], ck[VE];
#pragma unroll
          for (int e = 0; e < VE; e += 4) {
            *(float4*)&ca[e] = *(const float4*)&bn[4 * BNS + c0 + e];
            *(float4*)&cb[e] = *(const float4*)&bn[5 * BNS + c0 + e];
            *(float4*)&ck[e] = *(const float4*)&bn[6 * BNS + c0 + e];
          }
#pragma unroll
          for (int e = 0; e < VE; ++e) v[e] = fmaf(ca[e], St<T>::rnd(v[e]), fmaf(cb[e], z.v[e], ck[e]));
          if (P.res) {
            Chunk<T> x;
            unpack_chunk<T>(pre2[k], x);
#pragma unroll
            for (int e = 0; e < VE; ++e) v[e] += x.v[e];
          }
          store_chunk<T>(P.out, idx, v);
        } else {
          if (!(P.flags & EPI_NO_STORE)) store_chunk<T>(P.out, idx, v);
#pragma unroll
          for (int e = 0; e < VE; ++e) {
            const float dr = St<T>::rnd(v[e]);
            s1[e] += dr;
            s2[e] += dr * ((z.v[e] - mu[e]) * is[e]);
          }
        }
      } else {
        if (P.res) {
#pragma unroll
          for (int e = 0; e < VE; ++e) v[e] += pfc.v[e];
        }
        store_chunk<T>(P.out, idx, v);
      }
    }
  }

  const bool stats = (MODE == MODE_FWD) ? (P.flags & EPI_STATS) != 0 : (bnmask && !bnapply);
  if (stats) {
    __syncthreads();                   // acc_s reused: [rpp][BNc] sums, then sums of products
    float* red1 = acc_s;
    float* red2 = acc_s + 256 * VE;
    // row rr of the [rpp][BNc] sums keeps its 16-byte slots XOR-swizzled by bit (3 - log2 WN) of
    // rr, so that each half-wave's 16-byte writes fall on distinct banks
    constexpr int SWB = BNc == 64 ? 1 : BNc == 32 ? 2 : BNc == 16 ? 3 : 0;
    const int rr = tid / ncc;
#pragma unroll
    for (int e = 0; e < VE; e += 4) {
      const int slot = ((c0 + e) >> 2) ^ ((rr >> SWB) & 1);
      *(float4*)&red1[rr * BNc + slot * 4] = make_float4(s1[e], s1[e + 1], s1[e + 2], s1[e + 3]);
      *(float4*)&red2[rr * BNc + slot * 4] = make_float4(s2[e], s2[e + 1], s2[e + 2], s2[e + 3]);
    }
    __syncthreads();
    // column tid % BNc, row group tid / BNc: sums over the group's rows in order, then over the
    // groups in order
    constexpr int NQ = 256 / BNc;
    constexpr int RPQ = rpp / NQ;
    static_assert(NQ * RPQ == rpp && STAT_WORDS <= ACC_WORDS, "stats reduce layout");
    float* red3 = acc_s + 2 * 256 * VE;
    {
      const int col = tid % BNc, q = tid / BNc;
      float a = 0.f, b = 0.f;
#pragma unroll
      for (int k = q * RPQ; k < (q + 1) * RPQ; ++k) {
        const int w = k * BNc + ((((col >> 2) ^ ((k >> SWB) & 1))) << 2) + (col & 3);
        a += red1[w];
        b += red2[w];
      }
      red3[q * BNc + col] = a;
      red3[256 + q * BNc + col] = b;
    }
    __syncthreads();
    if (tid < BNc) {
      float a = 0.f, b = 0.f;
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        a += red3[q * BNc + tid];
        b += red3[256 + q * BNc + tid];
      }
      float2* pp = (float2*)P.part + (long)tm * P.ncol + n0 + tid;
      if (MODE == MODE_FWD) {
        // the tile's mean and sum of squared deviations from its pivoted sums (the pivot of column
        // tid as the threads that summed it formed it)
        const float n = (float)min(BM, P.M - tm * BM);
        const float am = a / n;
        st_coherent(pp, make_float2(piv_s[tid] + am, fmaxf(b - a * am, 0.f)));   // (read across XCDs)
      } else {
        *pp = make_float2(a, b);
      }
    }
    if (MODE == MODE_FWD && (P.flags & EPI_BN_FUSE))
      bn_fwd_fuse((float2*)P.part, P.tiles_m, BM, (long)P.M, P.ncol, P.bn_gamma, P.bn_stats, P.bn_cnt, tm, n0 / BNc,
                  n0, BNc, (double*)acc_s);
  }
}

}  // namespace pnn
