// BN forward statistics finalised by the kernel that produces their partial rows, instead of a
// separate column-reduce launch (training-mode BN of the layers H_l, Sec. 4).
#pragma once
#include "device_common.h"
#include "pnn_internal.h"

namespace pnn {

// part[r][c] (r < rows, c < C, stored with st_coherent) holds the mean and the sum of squared deviations of partial row r's
// n_r = min(rowh, count - r * rowh) rows of channel c.  Rows form groups of BNF_GROUP (the last
// group takes the remainder; a single group when rows < 2 BNF_GROUP).  Called by all 256 threads of
// a workgroup right after it wrote row tm, columns [c0, c0 + ncl) (column tile ct): the workgroup
// that completes a (group, column tile) folds the group's rows in fp64, in row order, into
// A = sum n_r mean_r and Q = sum (M2_r + n_r mean_r^2), kept as two doubles in place of the
// group's first two rows; the one that completes the column tile's last group adds the groups in
// group order and writes mean, invstd, scale = gamma invstd, shift = beta - mean scale ([4][C],
// the column-reduce kernel's finalisation).  Arrival counters cnt[ct][group], cnt[ct][groups] (each
// BNF_STRIDE words apart) are
// zero when the launch starts and are left zero.  Ordering: coherent stores, then each wave waits
// for its own (wait_mem) before the barrier that precedes the counter update; the reads follow the
// counter's result.  red: 512 doubles of LDS, free at the call.
__device__ __forceinline__ void bn_fwd_fuse(float2* part, int rows, int rowh, long count, int C, const float* gamma,
                                            float* stats, unsigned* cnt, int tm, int ct, int c0, int ncl,
                                            double* red) {
  __shared__ int bnf_last;
  const int tid = threadIdx.x;
  const int NG = (int)bnf_groups(rows);
  const int g = min(tm / BNF_GROUP, NG - 1);
  const int r0 = g * BNF_GROUP, r1 = g == NG - 1 ? rows : r0 + BNF_GROUP;
  unsigned* gc = cnt + (long)ct * (NG + 1) * BNF_STRIDE;
  wait_mem();                         // this workgroup's partial row, device-wide
  __syncthreads();
  if (tid == 0)
    bnf_last = __hip_atomic_fetch_add(&gc[g * BNF_STRIDE], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (unsigned)(r1 - r0 - 1);
  __syncthreads();
  if (!bnf_last) return;
  if (tid == 0) __hip_atomic_store(&gc[g * BNF_STRIDE], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const int CW = ncl < 256 ? ncl : 256;      // columns per pass
  const int LN = 256 / CW;                   // row lanes per column
  const int j = tid % CW, lane = tid / CW;
  double* dpart = (double*)part;
  auto finish = [&](int c, double A, double Q) {
    const double M = (double)count;
    const double mean = A / M;
    double var = Q / M - mean * mean;
    if (var < 0.0) var = 0.0;
    const float invstd = (float)(1.0 / sqrt(var + (double)PNN_BN_EPS));
    const float scale = gamma[c] * invstd;
    stats[c] = (float)mean;
    stats[C + c] = invstd;
    stats[2 * C + c] = scale;
    stats[3 * C + c] = gamma[C + c] - (float)mean * scale;
  };
  for (int cb = 0; cb < ncl; cb += CW) {
    const int c = c0 + cb + j;
    const bool on = lane < LN && cb + j < ncl;
    double A = 0.0, Q = 0.0;
    if (on) {
      int r = r0 + lane;
      for (; r + 3 * LN < r1; r += 4 * LN) {
        float2 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = ld_coherent(part + (long)(r + u * LN) * C + c);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const double n = (double)min((long)rowh, count - (long)(r + u * LN) * rowh), m = (double)v[u].x;
          A += n * m;
          Q += (double)v[u].y + n * m * m;
        }
      }
      for (; r < r1; r += LN) {
        const float2 v = ld_coherent(part + (long)r * C + c);
        const double n = (double)min((long)rowh, count - (long)r * rowh), m = (double)v.x;
        A += n * m;
        Q += (double)v.y + n * m * m;
      }
    }
    if (lane < LN) {
      red[lane * CW + j] = A;
      red[256 + lane * CW + j] = Q;
    }
    __syncthreads();
    if (lane == 0 && cb + j < ncl) {
      for (int k = 1; k < LN; ++k) {
        A += red[k * CW + j];
        Q += red[256 + k * CW + j];
      }
      if (NG == 1) {
        finish(c, A, Q);
      } else {
        st_coherent(dpart + (long)r0 * C + c, A);
        st_coherent(dpart + (long)(r0 + 1) * C + c, Q);
      }
    }
    __syncthreads();
  }
  if (NG == 1) return;
  wait_mem();                        // the group's (A, Q), device-wide
  __syncthreads();
  if (tid == 0)
    bnf_last = __hip_atomic_fetch_add(&gc[NG * BNF_STRIDE], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (unsigned)(NG - 1);
  __syncthreads();
  if (!bnf_last) return;
  if (tid == 0) __hip_atomic_store(&gc[NG * BNF_STRIDE], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  for (int cb = 0; cb < ncl; cb += CW) {
    const int c = c0 + cb + j;
    double A = 0.0, Q = 0.0;
    if (lane < LN && cb + j < ncl)
      for (int h = lane; h < NG; h += LN) {
        A += ld_coherent(dpart + (long)h * BNF_GROUP * C + c);
        Q += ld_coherent(dpart + ((long)h * BNF_GROUP + 1) * C + c);
      }
    if (lane < LN) {
      red[lane * CW + j] = A;
      red[256 + lane * CW + j] = Q;
    }
    __syncthreads();
    if (lane == 0 && cb + j < ncl) {
      for (int k = 1; k < LN; ++k) {
        A += red[k * CW + j];
        Q += red[256 + k * CW + j];
      }
      finish(c, A, Q);
    }
    __syncthreads();
  }
}

}  // namespace pnn
