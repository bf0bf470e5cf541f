// Normalisation, pooling, parareal-combine and head kernels for gfx950.
//
// BN (training mode, Sec. 4: the layers H_l of VGG-16 / ResNet-1001 are convolution, batch
// normalisation and ReLU) is split around the convolutions: its statistics are reduced from
// per-tile partial sums written by the producing kernel, and its affine map + ReLU is applied in
// the consuming kernel's operand load.  All reductions run in a fixed order (deterministic).
#include "bn_fuse.h"
#include "device_common.h"
#include "pnn_internal.h"

namespace pnn {

// ------------------------------------------------------------------------------------------------
// Column reduction of tile partials (split-K weight gradients, BN statistics, BN backward sums),
// fused with the BN finalisation.  A workgroup owns RED_COLS columns; its RED_LANES row lanes sum
// interleaved rows in fp64 and are combined in a fixed order (deterministic).
// ------------------------------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void colred_kernel(const ColRedLaunch L) {
  __shared__ double red[2 * RED_LANES][RED_COLS];   // RED_SUM uses all of it, BN modes the first half
  __shared__ double sum[RED_COLS];
  const int gi = find_group(L);
  const ColRedProb& P = L.p[gi];
  if (P.mode == RED_SUM) {
    // 2^rl_log2 row lanes x (1024 >> rl_log2) column pairs; lane l sums rows l, l + RL, ... in
    // order, then lane 0 adds the lanes' sums in lane order
    const int RL = 1 << P.rl_log2;
    const int CP = 1024 >> P.rl_log2;
    const int rl = threadIdx.x >> (10 - P.rl_log2);
    const int cp = threadIdx.x & (CP - 1);
    const int col = (blockIdx.x - P.tile_begin) * 2 * CP + 2 * cp;
    double a0 = 0.0, a1 = 0.0;
    if (col < P.ncols) {
      const float* p = P.part + col;
      int r = rl;
      for (; r + 3 * RL < P.rows; r += 4 * RL) {
        float2 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = *(const float2*)(p + (long)(r + u * RL) * P.ncols);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          a0 += (double)v[u].x;
          a1 += (double)v[u].y;
        }
      }
      for (; r < P.rows; r += RL) {
        const float2 v = *(const float2*)(p + (long)r * P.ncols);
        a0 += (double)v.x;
        a1 += (double)v.y;
      }
    }
    double* red2 = &red[0][0];
    red2[2 * threadIdx.x] = a0;
    red2[2 * threadIdx.x + 1] = a1;
    __syncthreads();
    if (rl == 0 && col < P.ncols) {
      for (int k = 1; k < RL; ++k) {
        a0 += red2[2 * (k * CP + cp)];
        a1 += red2[2 * (k * CP + cp) + 1];
      }
      P.dst[col] = (float)a0;
      P.dst[col + 1] = (float)a1;
    }
    return;
  }
  if (P.mode == RED_BN_FWD) {
    // partial row r holds, per channel, the mean and the sum of squared deviations of its n_r rows
    // (rows of rowh, the last one ragged).  In fp64, fixed order: A = sum_r n_r mean_r,
    // Q = sum_r (M2_r + n_r mean_r^2); mean = A / M, var = Q / M - mean^2 (exact up to fp64
    // rounding: the partial means carry the large part, the fp32 sums only the deviations)
    constexpr int CH = RED_COLS / 2, RLN = 1024 / CH;
    double (*ra)[CH] = (double (*)[CH])&red[0][0];
    double (*rq)[CH] = (double (*)[CH])&red[RLN / 2][0];
    const int C = P.ncols / 2;
    const int cl = threadIdx.x % CH, rl = threadIdx.x / CH;
    const int c = (blockIdx.x - P.tile_begin) * CH + cl;
    const float2* pp = (const float2*)P.part + c;
    const long h = P.rowh;
    double a = 0.0, q = 0.0;
    if (c < C) {
      int r = rl;
      for (; r + 3 * RLN < P.rows; r += 4 * RLN) {
        float2 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = pp[(long)(r + u * RLN) * C];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const double n = (double)min(h, P.count - (long)(r + u * RLN) * h), m = (double)v[u].x;
          a += n * m;
          q += (double)v[u].y + n * m * m;
        }
      }
      for (; r < P.rows; r += RLN) {
        const float2 v = pp[(long)r * C];
        const double n = (double)min(h, P.count - (long)r * h), m = (double)v.x;
        a += n * m;
        q += (double)v.y + n * m * m;
      }
    }
    // ra / rq: [RLN][CH] doubles each; red holds 2 * RED_LANES * RED_COLS = 2 * RLN * CH doubles
    ra[rl][cl] = a;
    rq[rl][cl] = q;
    __syncthreads();
#pragma unroll
    for (int k = RLN / 2; k >= 1; k >>= 1) {
      if (rl < k) {
        ra[rl][cl] += ra[rl + k][cl];
        rq[rl][cl] += rq[rl + k][cl];
      }
      __syncthreads();
    }
    if (rl != 0 || c >= C) return;
    const double M = (double)P.count;
    const double mean = ra[0][cl] / M;
    double var = rq[0][cl] / M - mean * mean;
    if (var < 0.0) var = 0.0;
    const float invstd = (float)(1.0 / sqrt(var + (double)PNN_BN_EPS));
    const float scale = P.gamma[c] * invstd;
    P.stats[c] = (float)mean;
    P.stats[C + c] = invstd;
    P.stats[2 * C + c] = scale;
    P.stats[3 * C + c] = P.beta[c] - (float)mean * scale;
    return;
  }
  const int c0 = (blockIdx.x - P.tile_begin) * RED_COLS;
  const int cl = threadIdx.x % RED_COLS;
  const int rl = threadIdx.x / RED_COLS;
  const int col = c0 + cl;
  double acc = 0.0;
  if (col < P.ncols) {
    // row lane rl sums rows rl, rl + S, ... with eight loads in flight (eight interleaved partial
    // sums, combined in a fixed order)
    const float* p = P.part + col;
    constexpr int S = RED_LANES;
    double a[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) a[u] = 0.0;
    int r = rl;
    for (; r + 7 * S < P.rows; r += 8 * S) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = p[(long)(r + u * S) * P.ncols];
#pragma unroll
      for (int u = 0; u < 8; ++u) a[u] += (double)v[u];
    }
    for (; r < P.rows; r += S) a[0] += (double)p[(long)r * P.ncols];
    acc = ((a[0] + a[1]) + (a[2] + a[3])) + ((a[4] + a[5]) + (a[6] + a[7]));
  }
  red[rl][cl] = acc;
  __syncthreads();
  // pairwise tree over the row lanes (fixed pairing)
#pragma unroll
  for (int h = RED_LANES / 2; h >= 1; h >>= 1) {
    if (rl < h) red[rl][cl] += red[rl + h][cl];
    __syncthreads();
  }
  if (rl == 0) sum[cl] = red[0][cl];
  __syncthreads();
  if (rl != 0 || col >= P.ncols) return;
  // BN modes: column 2c holds the first sum of channel c, column 2c+1 the second
  if (cl & 1) return;
  const int C = P.ncols / 2;
  const int c = col / 2;
  const double s1 = sum[cl], s2 = sum[cl + 1];
  const double M = (double)P.count;
  {
    // dL/dz = c1 (dbn - mb - xhat mbx), xhat = (z - mean) invstd, c1 = gamma invstd, mb = sum dbn / M,
    // mbx = sum dbn xhat / M; written as A dbn + B z + K per channel
    P.dbeta[c] = (float)s1;
    P.dgamma[c] = (float)s2;
    const double invstd = (double)P.stats[C + c], mean = (double)P.stats[c];
    const double c1 = (double)P.gamma[c] * invstd;
    const double mb = s1 / M, mbx = s2 / M;
    P.coef[c] = (float)c1;
    P.coef[C + c] = (float)(-c1 * mbx * invstd);
    P.coef[2 * C + c] = (float)(c1 * (mbx * invstd * mean - mb));
  }
}

// Column sums / sums of squares of a stored tensor [M][C], COLSTAT_ROWS rows per workgroup.
template <typename T>
__global__ __launch_bounds__(256) void colstat_kernel(const ColStatLaunch L) {
  // thread = (row lane, 16-byte column chunk); a lane sums its rows in order, lanes are added in
  // lane order through LDS
  constexpr int VE = St<T>::VE;
  __shared__ float2 red[256 * VE];
  const int gi = find_group(L);
  const ColStatProb& P = L.p[gi];
  const int tile = blockIdx.x - P.tile_begin;
  const long r0 = (long)tile * COLSTAT_ROWS;
  const long r1 = min(P.M, r0 + COLSTAT_ROWS);
  const int ncc = P.C / VE;
  const int RL = 256 / ncc;
  const int cc = threadIdx.x % ncc, rl = threadIdx.x / ncc;
  // sums about a pivot, the workgroup's first row, so that they do not cancel when a channel's mean
  // is large against its spread
  float s1[VE], s2[VE], pv[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) s1[e] = s2[e] = 0.f;
  {
    Chunk<T> c;
    load_chunk<T>(P.x, r0 * P.C + cc * VE, c);
#pragma unroll
    for (int e = 0; e < VE; ++e) pv[e] = c.v[e];
  }
  if (rl < RL) {
    long r = r0 + rl;
    for (; r + 3 * RL < r1; r += 4 * RL) {
      uint4 u[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) u[k] = *(const uint4*)((const T*)P.x + (r + k * RL) * P.C + cc * VE);
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        Chunk<T> c;
        unpack_chunk<T>(u[k], c);
#pragma unroll
        for (int e = 0; e < VE; ++e) {
          const float d = c.v[e] - pv[e];
          s1[e] += d;
          s2[e] += d * d;
        }
      }
    }
    for (; r < r1; r += RL) {
      Chunk<T> c;
      load_chunk<T>(P.x, r * P.C + cc * VE, c);
#pragma unroll
      for (int e = 0; e < VE; ++e) {
        const float d = c.v[e] - pv[e];
        s1[e] += d;
        s2[e] += d * d;
      }
    }
#pragma unroll
    for (int e = 0; e < VE; ++e) red[rl * P.C + cc * VE + e] = make_float2(s1[e], s2[e]);
  }
  __syncthreads();
  for (int c = threadIdx.x; c < P.C; c += 256) {
    float a = 0.f, b = 0.f;
    for (int k = 0; k < RL; ++k) {
      const float2 v = red[k * P.C + c];
      a += v.x;
      b += v.y;
    }
    // the workgroup's mean and sum of squared deviations
    const float am = a / (float)(r1 - r0);
    st_coherent((float2*)P.part + (long)tile * P.C + c, make_float2(St<T>::ld(P.x, r0 * P.C + c) + am, fmaxf(b - a * am, 0.f)));
  }
  if (P.fuse)
    bn_fwd_fuse((float2*)P.part, (int)((P.M + COLSTAT_ROWS - 1) / COLSTAT_ROWS), COLSTAT_ROWS, P.M, P.C, P.gamma,
                P.stats, P.cnt, tile, 0, 0, P.C, (double*)red);
}

// out = A dbn + B z + K [+ skip] per channel (the BN backward, coefficients from the column
// reduce); 16-byte chunks, C a multiple of the chunk.
template <typename T>
__global__ __launch_bounds__(256) void bn_apply_kernel(const BnApplyLaunch L) {
  constexpr int VE = St<T>::VE;
  const int gi = find_group(L);
  const BnApplyProb& P = L.p[gi];
  const long base = (long)(blockIdx.x - P.tile_begin) * ELT_TILE;
  for (int t = threadIdx.x * VE; t < ELT_TILE; t += 256 * VE) {
    const long i = base + t;
    if (i >= P.n) break;
    const int c0 = (int)(i % P.C);
    Chunk<T> d, z;
    load_chunk<T>(P.dbn, i, d);
    load_chunk<T>(P.z, i, z);
    float v[VE];
#pragma unroll
    for (int e = 0; e < VE; ++e)
      v[e] = fmaf(P.coef[c0 + e], d.v[e], fmaf(P.coef[P.C + c0 + e], z.v[e], P.coef[2 * P.C + c0 + e]));
    if (P.skip) {
      Chunk<T> k;
      load_chunk<T>(P.skip, i, k);
#pragma unroll
      for (int e = 0; e < VE; ++e) v[e] += k.v[e];
    }
    store_chunk<T>(P.out, i, v);
  }
}

// ------------------------------------------------------------------------------------------------
// SGD with momentum (Nesterov optional) and weight decay over a list of parameter tensors; every
// thread updates 8 consecutive elements of one tensor (16-byte / 32-byte vector accesses).
// ------------------------------------------------------------------------------------------------
__device__ __forceinline__ void sgd_elem(float& w, float g, float& v, float lr, float mu, float wd, bool nest) {
  const float d = fmaf(wd, w, g);
  v = fmaf(mu, v, d);
  const float u = nest ? fmaf(mu, v, d) : v;
  w = fmaf(-lr, u, w);
}

template <typename T>
__global__ __launch_bounds__(256) void sgd_kernel(const SgdLaunch L) {
  const int t = blockIdx.x;
  int lo = 0, hi = L.nt - 1;
  while (lo < hi) {                    // last entry with chunk0 <= t
    const int mid = (lo + hi + 1) >> 1;
    if ((int)L.e[mid].chunk0 <= t) lo = mid;
    else hi = mid - 1;
  }
  const SgdEnt& E = L.e[lo];
  const long i0 = (long)(t - (int)E.chunk0) * SGD_CHUNK + threadIdx.x * 8;
  if (i0 >= (long)E.count) return;
  char* pb = (char*)L.p[E.seg] + E.p_off;
  const float* gb = (const float*)((const char*)L.g[E.seg] + E.g_off) + i0;
  float* vb = (float*)((char*)L.v[E.seg] + E.g_off) + i0;
  const bool nest = L.nesterov != 0;
  const int n = (int)min((long)8, (long)E.count - i0);
  // fp32 master copy of a storage-type (bf16) filter: the update runs on it and the stored filter
  // is its rounding to nearest even, so updates below half a bf16 ulp accumulate
  float* mb = (!E.f32 && sizeof(T) == 2 && L.m[E.seg] != nullptr)
                  ? (float*)((char*)L.m[E.seg] + E.g_off) + i0 : nullptr;
  const bool from_master = mb != nullptr && !L.init;
  float w[8], g[8], v[8];
  if (n == 8) {
    const float4 g0 = *(const float4*)gb, g1 = *(const float4*)(gb + 4);
    const float4 v0 = *(const float4*)vb, v1 = *(const float4*)(vb + 4);
    g[0] = g0.x; g[1] = g0.y; g[2] = g0.z; g[3] = g0.w; g[4] = g1.x; g[5] = g1.y; g[6] = g1.z; g[7] = g1.w;
    v[0] = v0.x; v[1] = v0.y; v[2] = v0.z; v[3] = v0.w; v[4] = v1.x; v[5] = v1.y; v[6] = v1.z; v[7] = v1.w;
    if (E.f32 || sizeof(T) == 4 || from_master) {
      const float* wp = from_master ? mb : (const float*)pb + i0;
      const float4 w0 = *(const float4*)wp, w1 = *(const float4*)(wp + 4);
      w[0] = w0.x; w[1] = w0.y; w[2] = w0.z; w[3] = w0.w; w[4] = w1.x; w[5] = w1.y; w[6] = w1.z; w[7] = w1.w;
    } else {
      Chunk<uint16_t> c;
      load_chunk<uint16_t>(pb, i0, c);
#pragma unroll
      for (int e = 0; e < 8; ++e) w[e] = c.v[e];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) sgd_elem(w[e], g[e], v[e], L.lr, L.mu, L.wd, nest);
    *(float4*)vb = make_float4(v[0], v[1], v[2], v[3]);
    *(float4*)(vb + 4) = make_float4(v[4], v[5], v[6], v[7]);
    if (E.f32 || sizeof(T) == 4) {
      float* wp = (float*)pb + i0;
      *(float4*)wp = make_float4(w[0], w[1], w[2], w[3]);
      *(float4*)(wp + 4) = make_float4(w[4], w[5], w[6], w[7]);
    } else {
      store_chunk<uint16_t>(pb, i0, w);
      if (mb != nullptr) {
        *(float4*)mb = make_float4(w[0], w[1], w[2], w[3]);
        *(float4*)(mb + 4) = make_float4(w[4], w[5], w[6], w[7]);
      }
    }
    return;
  }
  for (int e = 0; e < n; ++e) {        // tail of the tensor
    float we = (E.f32 || sizeof(T) == 4) ? ((const float*)pb)[i0 + e]
               : from_master ? mb[e] : St<uint16_t>::ld(pb, i0 + e);
    float ve = vb[e];
    sgd_elem(we, gb[e], ve, L.lr, L.mu, L.wd, nest);
    vb[e] = ve;
    if (E.f32 || sizeof(T) == 4) {
      ((float*)pb)[i0 + e] = we;
    } else {
      St<uint16_t>::st(pb, i0 + e, we);
      if (mb != nullptr) mb[e] = we;
    }
  }
}

// ------------------------------------------------------------------------------------------------
// bnact: out = pool(ReLU(BN(z))) [+ res] [+ ext]; backward routes the output gradient to the first
// maximum of each 2x2 window, masks it by ReLU' and reduces dbn, dbn * xhat per channel.
// One workgroup = P.pix output pixels x all channels.  With C a multiple of the 16-byte chunk (VE
// elements) and at most BNACT_MAXC, a thread owns 16-byte chunks of channels (per-channel constants
// in LDS): forward work items are (pixel, chunk) pairs, several in flight per thread; backward, the
// 256 threads are (pixel lane, chunk) pairs, each lane summing its pixels' dbn, dbn * xhat, the
// lanes added in lane order.  Otherwise a thread owns channels, element by element.
// ------------------------------------------------------------------------------------------------
template <typename T>
__device__ __forceinline__ long bnact_zi(const BnActProb& P, long px, int Ho, int Wo, int pool, int w, int ch) {
  const int n = (int)(px / ((long)Ho * Wo));
  const int rem = (int)(px - (long)n * Ho * Wo);
  const int p = rem / Wo, q = rem - (rem / Wo) * Wo;
  return (((long)n * P.H + p * pool + w / pool) * P.W + q * pool + w % pool) * P.C + ch;
}

template <typename T>
__global__ __launch_bounds__(256) void bnact_fwd_kernel(const BnActLaunch L) {
  constexpr int VE = St<T>::VE;
  constexpr int U = 4;                                  // work items in flight per thread
  __shared__ float2 ss[BNACT_MAXC];                     // scale, shift per channel
  const int gi = find_group(L);
  const BnActProb& P = L.p[gi];
  const int pool = P.pool ? 2 : 1;
  const int Ho = P.H / pool, Wo = P.W / pool;
  const long px0 = (long)(blockIdx.x - P.tile_begin) * P.pix;
  const int tid = threadIdx.x;
  if (P.C % VE != 0 || P.C > BNACT_MAXC) {
    for (int c = tid; c < P.C; c += 256) {
      const float sc = P.stats[2 * P.C + c], sh = P.stats[3 * P.C + c];
      for (int k = 0; k < P.pix; ++k) {
        const long px = px0 + k;
        if (px >= P.n_out) break;
        float m = -INFINITY;
        for (int w = 0; w < pool * pool; ++w)
          m = fmaxf(m, fmaxf(fmaf(St<T>::ld(P.z, bnact_zi<T>(P, px, Ho, Wo, pool, w, c)), sc, sh), 0.0f));
        const long oi = px * P.C + c;
        if (P.res) m += St<T>::ld(P.res, oi);
        if (P.ext) m += St<T>::ld(P.ext, oi);
        St<T>::st(P.out, oi, m);
      }
    }
    return;
  }
  for (int c = tid; c < P.C; c += 256) ss[c] = make_float2(P.stats[2 * P.C + c], P.stats[3 * P.C + c]);
  __syncthreads();
  const int CC = P.C / VE;
  const int items = P.pix * CC;
  const int npool = pool * pool;
  for (int i0 = tid; i0 < items; i0 += 256 * U) {
    uint4 zv[U][4], rv[U], xv[U];
    long pxs[U];
    int chs[U];
    bool on[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int it = i0 + u * 256;
      pxs[u] = px0 + it / CC;
      chs[u] = (it % CC) * VE;
      on[u] = it < items && pxs[u] < P.n_out;
      const long px = on[u] ? pxs[u] : px0;
#pragma unroll
      for (int w = 0; w < 4; ++w)
        zv[u][w] = w < npool ? *(const uint4*)((const T*)P.z + bnact_zi<T>(P, px, Ho, Wo, pool, w, chs[u]))
                             : make_uint4(0, 0, 0, 0);
      const long oi = px * P.C + chs[u];
      rv[u] = P.res ? *(const uint4*)((const T*)P.res + oi) : make_uint4(0, 0, 0, 0);
      xv[u] = P.ext ? *(const uint4*)((const T*)P.ext + oi) : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (!on[u]) continue;
      float m[VE];
#pragma unroll
      for (int e = 0; e < VE; ++e) m[e] = -INFINITY;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        if (w >= npool) break;
        Chunk<T> z;
        unpack_chunk<T>(zv[u][w], z);
#pragma unroll
        for (int e = 0; e < VE; ++e) {
          const float2 q = ss[chs[u] + e];
          m[e] = fmaxf(m[e], fmaxf(fmaf(z.v[e], q.x, q.y), 0.0f));
        }
      }
      if (P.res) {
        Chunk<T> r;
        unpack_chunk<T>(rv[u], r);
#pragma unroll
        for (int e = 0; e < VE; ++e) m[e] += r.v[e];
      }
      if (P.ext) {
        Chunk<T> x;
        unpack_chunk<T>(xv[u], x);
#pragma unroll
        for (int e = 0; e < VE; ++e) m[e] += x.v[e];
      }
      store_chunk<T>(P.out, pxs[u] * P.C + chs[u], m);
    }
  }
}

template <typename T>
__global__ __launch_bounds__(256) void bnact_bwd_kernel(const BnActLaunch L) {
  constexpr int VE = St<T>::VE;
  __shared__ float4 cs[BNACT_MAXC];                     // mean, invstd, scale, shift per channel
  __shared__ float2 red[256 * VE];                      // per-lane sums [lanes][C]
  const int gi = find_group(L);
  const BnActProb& P = L.p[gi];
  const int pool = P.pool ? 2 : 1;
  const int Ho = P.H / pool, Wo = P.W / pool;
  const int npool = pool * pool;
  const int tile = blockIdx.x - P.tile_begin;
  const long px0 = (long)tile * P.pix;
  const int tid = threadIdx.x;
  if (P.C % VE != 0 || P.C > BNACT_MAXC) {
    for (int c = tid; c < P.C; c += 256) {
      const float mean = P.stats[c], invstd = P.stats[P.C + c];
      const float sc = P.stats[2 * P.C + c], sh = P.stats[3 * P.C + c];
      float s1 = 0.f, s2 = 0.f;
      for (int k = 0; k < P.pix; ++k) {
        const long px = px0 + k;
        if (px >= P.n_out) break;
        // first maximum of the window (row-major), on the unrounded activation
        int arg = 0;
        float best = 0.f;
        for (int w = 0; w < npool; ++w) {
          const float y = fmaxf(fmaf(St<T>::ld(P.z, bnact_zi<T>(P, px, Ho, Wo, pool, w, c)), sc, sh), 0.0f);
          if (w == 0 || y > best) {
            best = y;
            arg = w;
          }
        }
        const float gv = St<T>::ld(P.g, px * P.C + c);
        for (int w = 0; w < npool; ++w) {
          const long zi = bnact_zi<T>(P, px, Ho, Wo, pool, w, c);
          const float z = St<T>::ld(P.z, zi);
          const float y = fmaf(z, sc, sh);
          const float d = (w == arg && y > 0.f) ? gv : 0.f;
          St<T>::st(P.out, zi, d);
          const float dr = St<T>::rnd(d);
          s1 += dr;
          s2 += dr * ((z - mean) * invstd);
        }
      }
      ((float2*)P.part)[(long)tile * P.C + c] = make_float2(s1, s2);
    }
    return;
  }
  for (int c = tid; c < P.C; c += 256)
    cs[c] = make_float4(P.stats[c], P.stats[P.C + c], P.stats[2 * P.C + c], P.stats[3 * P.C + c]);
  __syncthreads();
  const int CC = P.C / VE;                              // chunks per pixel (<= 256 / 1 for C <= BNACT_MAXC)
  const int PL = 256 / CC;                              // pixel lanes
  const int cc = tid % CC, pl = tid / CC;
  const int ch = cc * VE;
  float s1[VE], s2[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) s1[e] = s2[e] = 0.f;
  if (pl < PL) {
#pragma unroll 2
    for (int k = pl; k < P.pix; k += PL) {
      const long px = px0 + k;
      if (px >= P.n_out) break;
      uint4 zv[4];
      long zi[4];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        zi[w] = bnact_zi<T>(P, px, Ho, Wo, pool, w < npool ? w : 0, ch);
        zv[w] = w < npool ? *(const uint4*)((const T*)P.z + zi[w]) : make_uint4(0, 0, 0, 0);
      }
      Chunk<T> g;
      unpack_chunk<T>(*(const uint4*)((const T*)P.g + px * P.C + ch), g);
      Chunk<T> z[4];
#pragma unroll
      for (int w = 0; w < 4; ++w) unpack_chunk<T>(zv[w], z[w]);
      // first maximum of each channel's window (row-major), on the unrounded activation
      int arg[VE];
#pragma unroll
      for (int e = 0; e < VE; ++e) {
        const float4 q = cs[ch + e];
        float best = 0.f;
        arg[e] = 0;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
          if (w >= npool) break;
          const float y = fmaxf(fmaf(z[w].v[e], q.z, q.w), 0.0f);
          if (w == 0 || y > best) {
            best = y;
            arg[e] = w;
          }
        }
      }
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        if (w >= npool) break;
        float d[VE];
#pragma unroll
        for (int e = 0; e < VE; ++e) {
          const float4 q = cs[ch + e];
          const float y = fmaf(z[w].v[e], q.z, q.w);
          d[e] = (w == arg[e] && y > 0.f) ? g.v[e] : 0.f;
          const float dr = St<T>::rnd(d[e]);
          s1[e] += dr;
          s2[e] += dr * ((z[w].v[e] - q.x) * q.y);
        }
        store_chunk<T>(P.out, zi[w], d);
      }
    }
#pragma unroll
    for (int e = 0; e < VE; ++e) red[pl * P.C + ch + e] = make_float2(s1[e], s2[e]);
  }
  __syncthreads();
  for (int c = tid; c < P.C; c += 256) {
    float a = 0.f, b = 0.f;
    for (int l = 0; l < PL; ++l) {
      a += red[l * P.C + c].x;
      b += red[l * P.C + c].y;
    }
    ((float2*)P.part)[(long)tile * P.C + c] = make_float2(a, b);
  }
}

// 3x3 / stride 2 / pad 1 max pool (preprocessing operators C^j, Sec. 4.1.1 and 4.2.1).  Each thread
// computes P.ve consecutive outputs of one pixel: a 16-byte chunk of channels (P.ve = elements per
// chunk; the host checks the channel count and alignment), or one element (P.ve = 1).
template <typename T>
__global__ __launch_bounds__(256) void maxpool3_kernel(const MaxPool3Launch L) {
  constexpr int VE = St<T>::VE;
  const int gi = find_group(L);
  const MaxPool3Prob& P = L.p[gi];
  const long n_out = (long)P.B * P.Ho * P.Wo * P.C;
  const bool vec = P.ve == VE;
  const long i = ((long)(blockIdx.x - P.tile_begin) * 256 + threadIdx.x) * P.ve;
  if (i >= n_out) return;
  const int c = (int)(i % P.C);
  const long px = i / P.C;
  const int q = (int)(px % P.Wo);
  const long np = px / P.Wo;
  const int p = (int)(np % P.Ho);
  const int n = (int)(np / P.Ho);
  float m[VE];
#pragma unroll
  for (int v = 0; v < VE; ++v) m[v] = -INFINITY;
#pragma unroll
  for (int a = 0; a < 3; ++a) {
    const int ih = 2 * p + a - 1;
#pragma unroll
    for (int b = 0; b < 3; ++b) {
      const int iw = 2 * q + b - 1;
      if (ih < 0 || ih >= P.H || iw < 0 || iw >= P.W) continue;
      const long src = (((long)n * P.H + ih) * P.W + iw) * P.C + c;
      if (vec) {
        Chunk<T> ch;
        load_chunk<T>(P.x, src, ch);
#pragma unroll
        for (int v = 0; v < VE; ++v) m[v] = fmaxf(m[v], ch.v[v]);
      } else {
        m[0] = fmaxf(m[0], St<T>::ld(P.x, src));
      }
    }
  }
  if (vec)
    store_chunk<T>(P.y, i, m);
  else
    St<T>::st(P.y, i, m[0]);
}

// wt[c][t][o] = w[o][t][c]  (filter layout of the data-gradient convolution): per tap, 64 x 64
// tiles of [o][c] through LDS so that reads and writes are both coalesced.  Tiles of a problem:
// T * ceil(O / 64) * ceil(C / 64), tap fastest.
template <typename T>
__global__ __launch_bounds__(256) void transpose_kernel(const TransposeLaunch L) {
  __shared__ T tile[64][65];
  const int gi = find_group(L);
  const TransposeProb& P = L.p[gi];
  const int lt = blockIdx.x - P.tile_begin;
  const int tp = lt % P.T;
  const int rest = lt / P.T;
  const int tiles_o = (P.O + 63) / 64;
  const int o0 = (rest % tiles_o) * 64, c0 = (rest / tiles_o) * 64;
  const T* w = (const T*)P.w;
  T* wt = (T*)P.wt;
  for (int k = threadIdx.x; k < 64 * 64; k += 256) {
    const int r = k >> 6, cc = k & 63;       // read w[o0 + r][tp][c0 + cc]
    if (o0 + r < P.O && c0 + cc < P.C) tile[r][cc] = w[((long)(o0 + r) * P.T + tp) * P.C + c0 + cc];
  }
  __syncthreads();
  for (int k = threadIdx.x; k < 64 * 64; k += 256) {
    const int r = k >> 6, oo = k & 63;       // write wt[c0 + r][tp][o0 + oo]
    if (c0 + r < P.C && o0 + oo < P.O) wt[((long)(c0 + r) * P.T + tp) * P.O + o0 + oo] = tile[oo][r];
  }
}

// out = a - b (rounded to storage); optional per-tile partial of sum(out^2) and non-finite flag.
// SUB_TILE elements per workgroup; a whole tile goes as 16-byte chunks with every load issued before
// the first store, a ragged last tile element by element.
template <typename T>
__global__ __launch_bounds__(256) void sub_kernel(const AxpyLaunch L) {
  constexpr int VE = St<T>::VE;
  constexpr int NCH = SUB_TILE / (256 * VE);          // chunks per thread
  __shared__ float red[4];
  const int gi = find_group(L);
  const AxpyProb& P = L.p[gi];
  const int tile = blockIdx.x - P.tile_begin;
  const long base = (long)tile * SUB_TILE;
  float sq = 0.f;
  bool bad = false;
  if (base + SUB_TILE <= P.n) {
    uint4 ua[NCH], ub[NCH];
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      const long i = base + (long)(k * 256 + threadIdx.x) * VE;
      ua[k] = *(const uint4*)((const T*)P.a + i);
      ub[k] = *(const uint4*)((const T*)P.b + i);
    }
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      const long i = base + (long)(k * 256 + threadIdx.x) * VE;
      Chunk<T> ca, cb;
      unpack_chunk<T>(ua[k], ca);
      unpack_chunk<T>(ub[k], cb);
      float v[VE];
#pragma unroll
      for (int e = 0; e < VE; ++e) {
        v[e] = ca.v[e] - cb.v[e];
        const float vr = St<T>::rnd(v[e]);
        sq += vr * vr;
        bad |= !isfinite(vr);
      }
      store_chunk<T>(P.out, i, v);
    }
  } else {
    for (int t = threadIdx.x; t < SUB_TILE; t += 256) {
      const long i = base + t;
      if (i >= P.n) break;
      const float v = St<T>::ld(P.a, i) - St<T>::ld(P.b, i);
      St<T>::st(P.out, i, v);
      const float vr = St<T>::rnd(v);
      sq += vr * vr;
      bad |= !isfinite(vr);
    }
  }
  if (L.flag != nullptr && __syncthreads_or(bad) && threadIdx.x == 0)
    __hip_atomic_store(L.flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (P.sq_part != nullptr) {
    sq = wave_sum(sq);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = sq;
    __syncthreads();
    if (threadIdx.x == 0) P.sq_part[tile] = ((red[0] + red[1]) + red[2]) + red[3];
  }
}

__global__ void sumsq_kernel(const float* part, int n, float* out) {
  if (threadIdx.x == 0 && blockIdx.x == 0) {
    double s = 0.0;
    for (int i = 0; i < n; ++i) s += part[i];
    *out = (float)s;
  }
}

// ------------------------------------------------------------------------------------------------
// head h: logits = mean_{hw}(ytilde) W^T + b, softmax cross-entropy (mean over the batch), and
// D_N = dL/dytilde.  Kernel 1: one workgroup per sample.  Kernel 2: dW, db, loss.  Every sum runs
// in an order fixed by the shapes alone, so repeated calls give identical bits.
// scratch: pooled [B][C], dlogits [B][K], loss_n [B]
// ------------------------------------------------------------------------------------------------
// G > 0: 16-byte chunks (C a multiple of the chunk), the pixels split over G row groups, each
// summing its pixels into part[g][C]; G = 0: one element per load, one row group.
template <typename T>
__global__ __launch_bounds__(256) void head_sample_kernel(const void* yt, const float* eps,
                                                          const int32_t* labels, float* logits,
                                                          void* D_N, float* scratch, int B, int HW,
                                                          int C, int K, int G) {
  extern __shared__ float sh[];  // pooled [C], z (then dlogits) [K], part [G][C] when G > 1
  constexpr int VE = St<T>::VE;
  float* pooled = sh;
  float* z = sh + C;
  float* part = G > 1 ? z + K : pooled;
  __shared__ float red[1];
  const int n = blockIdx.x, t = threadIdx.x, lane = t & 63, wave = t >> 6;
  const float* W = eps;
  const float* bias = eps + (long)K * C;
  const long base = (long)n * HW * C;
  const int GG = G > 0 ? G : 1;
  if (G > 0) {
    const int nch = C / VE;
    for (int i = t; i < G * nch; i += 256) {
      const int q = i % nch, g = i / nch;
      float acc[VE];
#pragma unroll
      for (int v = 0; v < VE; ++v) acc[v] = 0.f;
#pragma unroll 8
      for (int h = g; h < HW; h += G) {
        Chunk<T> ch;
        load_chunk<T>(yt, base + (long)h * C + q * VE, ch);
#pragma unroll
        for (int v = 0; v < VE; ++v) acc[v] += ch.v[v];
      }
#pragma unroll
      for (int v = 0; v < VE; ++v) part[g * C + q * VE + v] = acc[v];
    }
  } else {
    for (int c = t; c < C; c += 256) {
      float acc = 0.f;
      for (int h = 0; h < HW; ++h) acc += St<T>::ld(yt, base + (long)h * C + c);
      part[c] = acc;
    }
  }
  __syncthreads();
  for (int c = t; c < C; c += 256) {
    float acc = 0.f;
    for (int g = 0; g < GG; ++g) acc += part[g * C + c];
    pooled[c] = acc / (float)HW;
    scratch[(long)n * C + c] = pooled[c];
  }
  __syncthreads();
  // logits: wave w takes the classes 8 w .. 8 w + 7 (mod 32), its lanes stride over the channels
  for (int k0 = 8 * wave; k0 < K; k0 += 32) {
    float acc[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) acc[u] = 0.f;
#pragma unroll 4
    for (int c = lane; c < C; c += 64) {
      const float pc = pooled[c];
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (k0 + u < K) acc[u] += W[(long)(k0 + u) * C + c] * pc;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) acc[u] += __shfl_xor(acc[u], o);
    if (lane == 0)
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (k0 + u < K) {
          z[k0 + u] = acc[u] + bias[k0 + u];
          if (logits) logits[(long)n * K + k0 + u] = acc[u] + bias[k0 + u];
        }
  }
  __syncthreads();
  if (wave == 0) {  // log-sum-exp, the exponentials summed in double
    float mx = -INFINITY;
    for (int k = lane; k < K; k += 64) mx = fmaxf(mx, z[k]);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) mx = fmaxf(mx, __shfl_xor(mx, o));
    double se = 0.0;
    for (int k = lane; k < K; k += 64) se += exp((double)(z[k] - mx));
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) se += __shfl_xor(se, o);
    if (lane == 0) red[0] = mx + (float)log(se);
  }
  __syncthreads();
  const float lse = red[0];
  const int lab = labels[n];
  const bool lab_ok = lab >= 0 && lab < K;  // a label outside [0, K) gives a NaN loss
  if (t == 0) scratch[(long)B * C + (long)B * K + n] = lab_ok ? lse - z[lab] : NAN;
  __syncthreads();
  float* dlog = scratch + (long)B * C;
  for (int k = t; k < K; k += 256) {
    const float d = (expf(z[k] - lse) - (k == lab ? 1.f : 0.f)) / (float)B;
    z[k] = d;
    dlog[(long)n * K + k] = d;
  }
  __syncthreads();
  // D_N[n, h, c] = (sum_k dlogits[k] W[k, c]) / HW for every pixel h: per channel once (into the
  // pooled array, no longer needed), then stored over the pixels
  for (int c = t; c < C; c += 256) {
    float acc = 0.f;
#pragma unroll 32
    for (int k = 0; k < K; ++k) acc += z[k] * W[(long)k * C + c];
    pooled[c] = acc / (float)HW;
  }
  __syncthreads();
  if (G > 0) {
    const int nch = C / VE;
    for (int i = t; i < G * nch; i += 256) {
      const int q = i % nch, g = i / nch;
      float d[VE];
#pragma unroll
      for (int v = 0; v < VE; ++v) d[v] = pooled[q * VE + v];
      for (int h = g; h < HW; h += G) store_chunk<T>(D_N, base + (long)h * C + q * VE, d);
    }
  } else {
    for (int c = t; c < C; c += 256) {
      const float d = pooled[c];
      for (int h = 0; h < HW; ++h) St<T>::st(D_N, base + (long)h * C + c, d);
    }
  }
}

// 64 outputs of [dW | db | loss] per workgroup; wave w sums the samples of its quarter of the
// batch, the four partial sums are added in wave order.
__global__ __launch_bounds__(256) void head_reduce_kernel(const float* scratch, float* deps,
                                                          float* loss, int B, int C, int K, unsigned* flag) {
  __shared__ float rs[4][64];
  __shared__ double rl[4];
  const float* pooled = scratch;
  const float* dlog = scratch + (long)B * C;
  const float* ln = dlog + (long)B * K;
  const long nW = (long)K * C;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const long i = (long)blockIdx.x * 64 + lane;
  const int nb = (B + 3) / 4, n0 = wave * nb, n1 = min(B, n0 + nb);
  float acc = 0.f;
  if (i < nW) {
    const int k = (int)(i / C), c = (int)(i % C);
#pragma unroll 16
    for (int n = n0; n < n1; ++n) acc += dlog[(long)n * K + k] * pooled[(long)n * C + c];
  } else if (i < nW + K) {
    const int k = (int)(i - nW);
#pragma unroll 8
    for (int n = n0; n < n1; ++n) acc += dlog[(long)n * K + k];
  } else if (i == nW + K) {
    double sl = 0.0;
    for (int n = n0; n < n1; ++n) sl += ln[n];
    rl[wave] = sl;
  }
  rs[wave][lane] = acc;
  __syncthreads();
  bool bad = false;
  if (wave == 0) {
    if (i < nW + K) {
      const float v = ((rs[0][lane] + rs[1][lane]) + rs[2][lane]) + rs[3][lane];
      deps[i] = v;
      bad = !isfinite(v);
    } else if (i == nW + K) {
      const float v = (float)((((rl[0] + rl[1]) + rl[2]) + rl[3]) / (double)B);
      *loss = v;
      bad = !isfinite(v);
    }
  }
  if (flag != nullptr && __syncthreads_or(bad) && threadIdx.x == 0)
    __hip_atomic_store(flag, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__global__ void flags_clear_kernel(unsigned* flags) {
  if (threadIdx.x < PNN_NFLAGS) flags[threadIdx.x] = 0u;
}

// word ranges set to zero (arrival counters), ZERO_WORDS words per workgroup
__global__ __launch_bounds__(256) void zero_kernel(const ZeroLaunch L) {
  const int gi = find_group(L);
  const ZeroProb& P = L.p[gi];
  const int w0 = (blockIdx.x - P.tile_begin) * ZERO_WORDS;
  const int w1 = min(P.words, w0 + ZERO_WORDS);
  for (int w = w0 + (int)threadIdx.x; w < w1; w += 256) P.p[w] = 0u;
}

// ------------------------------------------------------------------------------------------------
// launchers
// ------------------------------------------------------------------------------------------------
#define PNN_LAUNCH_T(kern, L, tiles, dtype, s)                                        \
  do {                                                                               \
    if ((dtype) == 1)                                                                \
      hipLaunchKernelGGL(kern<uint16_t>, dim3(tiles), dim3(256), 0, s, L);           \
    else                                                                             \
      hipLaunchKernelGGL(kern<float>, dim3(tiles), dim3(256), 0, s, L);              \
    return (int)hipGetLastError();                                                   \
  } while (0)

int launch_colred(const ColRedLaunch& L, int tiles, hipStream_t s) {
  hipLaunchKernelGGL(colred_kernel, dim3(tiles), dim3(RED_COLS * RED_LANES), 0, s, L);
  return (int)hipGetLastError();
}
int launch_sgd(const SgdLaunch& L, int tiles, int dtype, hipStream_t s) {
  PNN_LAUNCH_T(sgd_kernel, L, tiles, dtype, s);
}
int launch_colstat(const ColStatLaunch& L, int tiles, int dtype, hipStream_t s) {
  PNN_LAUNCH_T(colstat_kernel, L, tiles, dtype, s);
}
int launch_bn_apply(const BnApplyLaunch& L, int tiles, int dtype, hipStream_t s) {
  PNN_LAUNCH_T(bn_apply_kernel, L, tiles, dtype, s);
}
int launch_bnact_fwd(const BnActLaunch& L, int tiles, int dtype, hipStream_t s) {
  PNN_LAUNCH_T(bnact_fwd_kernel, L, tiles, dtype, s);
}
int launch_bnact_bwd(const BnActLaunch& L, int tiles, int dtype, hipStream_t s) {
  PNN_LAUNCH_T(bnact_bwd_kernel, L, tiles, dtype, s);
}
int launch_maxpool3(const MaxPool3Launch& L, int tiles, int dtype, hipStream_t s) {
  PNN_LAUNCH_T(maxpool3_kernel, L, tiles, dtype, s);
}
int launch_transpose(const TransposeLaunch& L, int tiles, int dtype, hipStream_t s) {
  PNN_LAUNCH_T(transpose_kernel, L, tiles, dtype, s);
}
int launch_sub(const AxpyLaunch& L, int tiles, int dtype, hipStream_t s) {
  PNN_LAUNCH_T(sub_kernel, L, tiles, dtype, s);
}
int launch_zero(const ZeroLaunch& L, int tiles, hipStream_t s) {
  hipLaunchKernelGGL(zero_kernel, dim3(tiles), dim3(256), 0, s, L);
  return (int)hipGetLastError();
}
int launch_flags_clear(unsigned* flags, hipStream_t s) {
  hipLaunchKernelGGL(flags_clear_kernel, dim3(1), dim3(64), 0, s, flags);
  return (int)hipGetLastError();
}
int launch_sumsq(const float* part, int n, float* out, hipStream_t s) {
  hipLaunchKernelGGL(sumsq_kernel, dim3(1), dim3(64), 0, s, part, n, out);
  return (int)hipGetLastError();
}

int launch_head(const void* yt, const float* eps, const int32_t* labels, float* logits, float* loss,
                void* D_N, float* deps, float* scratch, int B, int HW, int C, int K, int dtype,
                unsigned* flag, hipStream_t s) {
  const int es = dtype == 1 ? 2 : 4, ve = 16 / es;
  const bool vec = C % ve == 0 && ((uintptr_t)yt % 16) == 0 && ((uintptr_t)D_N % 16) == 0;
  int G = 0;
  if (vec) {
    const int nch = C / ve;
    G = nch >= 256 ? 1 : std::max(1, std::min(256 / nch, HW));
  }
  const size_t shm = sizeof(float) * ((size_t)C + K + (G > 1 ? (size_t)G * C : 0));
  if (dtype == 1)
    hipLaunchKernelGGL(head_sample_kernel<uint16_t>, dim3(B), dim3(256), shm, s, yt, eps, labels,
                       logits, D_N, scratch, B, HW, C, K, G);
  else
    hipLaunchKernelGGL(head_sample_kernel<float>, dim3(B), dim3(256), shm, s, yt, eps, labels,
                       logits, D_N, scratch, B, HW, C, K, G);
  int e = (int)hipGetLastError();
  if (e) return e;
  const long n = (long)K * C + K + 1;
  hipLaunchKernelGGL(head_reduce_kernel, dim3((unsigned)((n + 63) / 64)), dim3(256), 0, s,
                     scratch, deps, loss, B, C, K, flag);
  return (int)hipGetLastError();
}

}  // namespace pnn
