// Grouped implicit-GEMM convolution kernels for gfx950 (forward, data gradient, weight gradient).
//
// Convolution, its data gradient and its weight gradient are the three contractions of every
// layer of the fine sub-networks g^j and coarse blocks F^j (Sec. 3, Alg. para2 / para3).  One
// launch runs the same layer position of all N sub-networks: every group is an independent
// problem with its own tensors and filters.
//
// Operands are NHWC rows gathered with 16-byte loads straight into MFMA lane fragments (bf16:
// v_mfma_f32_16x16x32_bf16, fp32: v_mfma_f32_16x16x4f32); accumulation is fp32.  A workgroup of
// four waves owns a 128-row x (16 wn)-column output tile; each wave 32 rows.
#include "device_common.h"
#include "pnn_internal.h"
#include "conv_epilogue.h"

namespace pnn {

// ------------------------------------------------------------------------------------------------
// forward / data-gradient convolution
//
// GK = gather kind: GK_POINT  1x1 / stride 1 / pad 0 (row m of A is row m of the input),
//                   GK_VEC    any geometry, channels a multiple of the 16-byte chunk,
//                   GK_SCALAR any geometry, element-wise gather (e.g. 3-channel images),
//                   GK_HALO   3x3 / stride 1 / pad 1 (forward, and its data gradient, which is the
//                             same stencil with the taps mirrored): the tile's input rows plus a
//                             one-pixel halo are staged in LDS once, the filter column of each wave
//                             is held in registers, and every K step reads A from LDS.
// The BN prologue's (scale, shift) and the data-gradient epilogue's BN statistics are staged in LDS
// once per workgroup.  The epilogue stages the fp32 tile through LDS so that every thread owns
// 16-byte column chunks: residual / mask-source loads and output stores are 16-byte vectors, and
// each thread's BN partial sums cover fixed columns (combined in a fixed order).
// ------------------------------------------------------------------------------------------------
enum { GK_POINT = 0, GK_VEC = 1, GK_SCALAR = 2, GK_HALO = 3 };

template <typename T, int MODE, int GK>
__device__ __forceinline__ void gather_a(const ConvProb& P, const float2* pro, int m, int n, int p, int q,
                                         bool rowok, int k0, Frag<T>& a) {
  constexpr int VE = St<T>::VE;
  const bool prologue = MODE == MODE_FWD && P.pro != nullptr;
  if constexpr (GK == GK_POINT) {
    if (!(rowok && k0 < P.K)) {
      a.zero();
      return;
    }
    const long idx = (long)m * P.Cg + k0;
    if (prologue) {
      Chunk<T> c;
      load_chunk<T>(P.in, idx, c);
#pragma unroll
      for (int e = 0; e < VE; ++e) c.v[e] = fmaxf(fmaf(c.v[e], pro[k0 + e].x, pro[k0 + e].y), 0.0f);
      a.from_chunk(c);
    } else {
      a.from_raw(*(const uint4*)((const T*)P.in + idx));
    }
  } else if constexpr (GK == GK_VEC) {
    const int tap = div_l2(k0, P.Cg, P.cg_log2);
    const int c0 = k0 - tap * P.Cg;
    int r, s;
    tap_rs(tap, P.k, r, s);
    int ih, iw;
    bool ok = rowok && k0 < P.K;
    if constexpr (MODE == MODE_FWD) {
      ih = p * P.stride + r - P.pad;
      iw = q * P.stride + s - P.pad;
    } else {
      const int th = p + P.pad - r, tw = q + P.pad - s;
      if (P.stride == 1) {
        ih = th;
        iw = tw;
      } else {   // stride 2
        ok = ok && th >= 0 && tw >= 0 && ((th | tw) & 1) == 0;
        ih = th >> 1;
        iw = tw >> 1;
      }
    }
    ok = ok && (unsigned)ih < (unsigned)P.H && (unsigned)iw < (unsigned)P.W;
    if (!ok) {
      a.zero();
      return;
    }
    const long idx = (((long)n * P.H + ih) * P.W + iw) * P.Cg + c0;
    if (prologue) {
      Chunk<T> c;
      load_chunk<T>(P.in, idx, c);
#pragma unroll
      for (int e = 0; e < VE; ++e) c.v[e] = fmaxf(fmaf(c.v[e], pro[c0 + e].x, pro[c0 + e].y), 0.0f);
      a.from_chunk(c);
    } else {
      a.from_raw(*(const uint4*)((const T*)P.in + idx));
    }
  } else {
    Chunk<T> c;
#pragma unroll
    for (int e = 0; e < VE; ++e) {
      const int kk = k0 + e;
      float v = 0.0f;
      if (rowok && kk < P.K) {
        const int tap = kk / P.Cg;
        const int ch = kk - tap * P.Cg;
        const int r = tap / P.k;
        const int s = tap - r * P.k;
        int ih, iw;
        bool ok = true;
        if constexpr (MODE == MODE_FWD) {
          ih = p * P.stride + r - P.pad;
          iw = q * P.stride + s - P.pad;
        } else {
          const int th = p + P.pad - r, tw = q + P.pad - s;
          ok = th >= 0 && tw >= 0 && (th % P.stride) == 0 && (tw % P.stride) == 0;
          ih = th / P.stride;
          iw = tw / P.stride;
        }
        ok = ok && (unsigned)ih < (unsigned)P.H && (unsigned)iw < (unsigned)P.W;
        if (ok) {
          v = St<T>::ld(P.in, (((long)n * P.H + ih) * P.W + iw) * P.Cg + ch);
          if (prologue) v = fmaxf(fmaf(v, pro[ch].x, pro[ch].y), 0.0f);
        }
      }
      c.v[e] = v;
    }
    a.from_chunk(c);
  }
}

template <typename T, bool VEC>
__device__ __forceinline__ void load_b(const ConvProb& P, int col, int k0, Frag<T>& b) {
  constexpr int VE = St<T>::VE;
  if constexpr (VEC) {
    if (k0 < P.K)
      b.from_raw(*(const uint4*)((const T*)P.wmat + (long)col * P.K + k0));
    else
      b.zero();
  } else {
    Chunk<T> c;
#pragma unroll
    for (int e = 0; e < VE; ++e)
      c.v[e] = (k0 + e < P.K) ? St<T>::ld(P.wmat, (long)col * P.K + k0 + e) : 0.0f;
    b.from_chunk(c);
  }
}


// GK_HALO main loop.  The tile's BM output rows are whole image rows (BM a multiple of Q): either
// R = BM / Q rows of one image or BM / PQ whole images.  LDS holds those rows plus a one-pixel halo
// of the (activated, for the forward prologue) input; padding pixels are zeros.  A pixel's Cg
// channels are followed by 0 or 2 unused 16-byte chunks (conv_halo_pad), a pixel stride that keeps
// each half-wave's A reads (16 pixels x an aligned chunk pair) on few shared LDS banks.  Wave w
// owns column sub-tile w % WN and WM * WN row sub-tiles; its filter fragments for all K steps (at most
// conv_halo_nkb(WN)) are loaded into registers before the LDS fill completes.  Steps past K read a
// valid A position; the filter fragment there is zero.
template <typename T, int MODE, int WM, int WN, typename F>
__device__ __forceinline__ void conv_halo(const ConvProb& P, const float2* pro, T* halo, int tm, int n0,
                                          f32x4 (&acc)[WM][WN], F&& before_compute) {
  constexpr int VE = St<T>::VE;
  constexpr int KS = 4 * VE;
  constexpr int BM = 64 * WM;
  constexpr int NT = WM * WN;                 // row sub-tiles per wave
  constexpr int NKB = conv_halo_nkb(WN);
  constexpr int NL = 8;                      // halo chunks in flight per thread
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int r16 = lane & 15, grp = lane >> 4;
  const int PQ = P.P * P.Q;
  const int QH = P.Q + 2;
  const int PS = P.Cg + conv_halo_pad(P.Cg / VE, P.Q) * VE;
  const bool multi = BM > PQ;
  const int R = multi ? P.P : BM / P.Q;
  const int RH = R + 2;
  const int nimg = multi ? BM / PQ : 1;
  const int m0 = tm * BM;
  const int n_first = div_l2(m0, PQ, P.pq_log2);
  const int p0 = multi ? 0 : div_l2(m0 - n_first * PQ, P.Q, P.q_log2);
  const int cpp = P.Cg / VE;
  const int img_px = RH * QH;
  const int total = nimg * img_px * cpp;
  const int ct = wave % WN, rg = wave / WN;
  const int nsteps = (P.K + KS - 1) / KS;

  Frag<T> bq[NKB];
#pragma unroll
  for (int s = 0; s < NKB; ++s) {
    if (s < nsteps) load_b<T, true>(P, n0 + ct * 16 + r16, s * KS + VE * grp, bq[s]);
    else bq[s].zero();
  }

  const float r_cpp = 1.0f / cpp, r_img = 1.0f / img_px, r_qh = 1.0f / QH;
  // one image per tile and a power-of-two chunk count per pixel (the usual case): shifts for the
  // chunk / pixel split and 32-bit offsets from the image's first element
  const int cpp_l2 = P.cg_log2 - (VE == 8 ? 3 : 2);
  const bool fast = nimg == 1 && cpp_l2 >= 0 && (long)P.H * P.W * P.Cg < (1L << 31);
  const T* img0 = (const T*)P.in + (long)n_first * P.H * P.W * P.Cg;
  for (int base = 0; base < total; base += 256 * NL) {
    uint4 v[NL];
    int off[NL], cv[NL];
    bool ok[NL];
#pragma unroll
    for (int u = 0; u < NL; ++u) {
      const int idx = base + u * 256 + tid;
      if (fast) {
        const int ch = idx & (cpp - 1), pix = idx >> cpp_l2;
        int y, x;
        divmod_small(pix, QH, r_qh, y, x);
        const int ih = p0 - 1 + y, iw = x - 1;
        ok[u] = idx < total && (unsigned)ih < (unsigned)P.H && (unsigned)iw < (unsigned)P.W;
        off[u] = idx < total ? pix * PS + ch * VE : -1;
        cv[u] = ch * VE;
        const int g = ok[u] ? ((ih * P.W + iw) << P.cg_log2) + ch * VE : 0;
        v[u] = *(const uint4*)(img0 + g);
        continue;
      }
      int pix, ch, i, rem, y, x;
      divmod_small(idx, cpp, r_cpp, pix, ch);
      if (nimg > 1) divmod_small(pix, img_px, r_img, i, rem);
      else { i = 0; rem = pix; }
      divmod_small(rem, QH, r_qh, y, x);
      const int n = n_first + i, ih = p0 - 1 + y, iw = x - 1;
      ok[u] = idx < total && n < P.B && (unsigned)ih < (unsigned)P.H && (unsigned)iw < (unsigned)P.W;
      off[u] = idx < total ? pix * PS + ch * VE : -1;
      cv[u] = ch * VE;
      const long g = ok[u] ? (((long)n * P.H + ih) * P.W + iw) * P.Cg + ch * VE : 0;
      v[u] = *(const uint4*)((const T*)P.in + g);
    }
#pragma unroll
    for (int u = 0; u < NL; ++u) {
      if (off[u] < 0) continue;
      uint4 w = make_uint4(0, 0, 0, 0);
      if (ok[u]) {
        if (MODE == MODE_FWD && P.pro != nullptr) {
          Chunk<T> c;
          unpack_chunk<T>(v[u], c);
          float f[VE];
#pragma unroll
          for (int e = 0; e < VE; ++e) f[e] = fmaxf(fmaf(c.v[e], pro[cv[u] + e].x, pro[cv[u] + e].y), 0.0f);
          store_chunk<T>(&w, 0, f);
        } else {
          w = v[u];
        }
      }
      *(uint4*)(halo + off[u]) = w;
    }
  }

  int rb[NT];                                  // LDS element offset of the sub-tile row's pixel
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const int lm = (rg * NT + t) * 16 + r16;
    const int i = multi ? div_l2(lm, PQ, P.pq_log2) : 0;
    const int rem = lm - i * R * P.Q;
    const int pl = div_l2(rem, P.Q, P.q_log2);
    const int ql = rem - pl * P.Q;
    rb[t] = ((i * RH + pl) * QH + ql) * PS;
  }
  __syncthreads();
  before_compute();                           // the epilogue's early loads overlap the K loop

#pragma unroll
  for (int s = 0; s < NKB; ++s) {
    if (s < nsteps) {
      int k0 = s * KS + VE * grp;
      if (k0 >= P.K) k0 = 0;
      const int tap = div_l2(k0, P.Cg, P.cg_log2);
      const int c0 = k0 - tap * P.Cg;
      int r, q;
      tap_rs(tap, 3, r, q);
      const int toff = ((MODE == MODE_FWD) ? (r * QH + q) : ((2 - r) * QH + (2 - q))) * PS + c0;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        Frag<T> a;
        a.from_raw(*(const uint4*)(halo + rb[t] + toff));
        mma(a, bq[s], acc[t / WN][t % WN]);
      }
    }
  }
  __syncthreads();                            // the halo region is reused by the epilogue
}

// WM row sub-tiles of 16 per wave, WN column sub-tiles: a workgroup owns a (64 WM) x (16 WN) tile
// (tall tiles: WM * WN = CONV_SUBTILES, so narrow problems get taller tiles; short tiles: 2 or 4).
template <typename T, int MODE, int GK, int WM, int WN>
__global__ __launch_bounds__(256) void conv_kernel(const ConvLaunch L) {
  constexpr int VE = St<T>::VE;
  constexpr int KS = 4 * VE;
  constexpr int BM = 64 * WM;
  constexpr int LDA = 16 * WN + 4;
  constexpr int STAT_WORDS = 2 * 256 * VE + 512;   // BN sums reduce (epilogue)
  constexpr int ACC_WORDS0 = BM * LDA > STAT_WORDS ? BM * LDA : STAT_WORDS;
  constexpr int ACC_WORDS = (GK == GK_HALO && CONV_HALO_BYTES / 4 > ACC_WORDS0) ? CONV_HALO_BYTES / 4 : ACC_WORDS0;
  // BN prologue constants (forward only) and BN statistics / apply coefficients (data gradient
  // only): each mode allocates only its own, which keeps four workgroups resident per CU
  __shared__ float2 pro_s[MODE == MODE_FWD ? CONV_PRO_MAXC : 1];
  __shared__ __attribute__((aligned(16))) float bn_s[MODE == MODE_BWD ? 7 : 1][64];   // mean, invstd, scale, shift; A, B, K
  __shared__ __attribute__((aligned(16))) float acc_s[ACC_WORDS];

  const int gi = find_group(L);
  const ConvProb& P = L.p[gi];
  const int local = blockIdx.x - P.tile_begin;
  const int tm = local / P.tiles_n;
  const int tn = local - tm * P.tiles_n;
  const int tid = threadIdx.x;
  const int wave = tid >> 6;
  const int lane = tid & 63;
  const int r16 = lane & 15;
  const int grp = lane >> 4;
  const int mw = tm * BM + wave * 16 * WM;
  const int n0 = tn * 16 * P.wn;
  const int PQ = P.P * P.Q;
  const bool bnmask = MODE == MODE_BWD && (P.flags & (EPI_BN_MASK | EPI_BN_APPLY));
  const bool bnapply = MODE == MODE_BWD && (P.flags & EPI_BN_APPLY);

  int rm[WM], rn[WM], rp[WM], rq[WM];
  bool rv[WM];
#pragma unroll
  for (int wm = 0; wm < WM && GK != GK_HALO; ++wm) {
    const int m = mw + wm * 16 + r16;
    rv[wm] = m < P.M;
    const int mm = rv[wm] ? m : 0;
    rm[wm] = mm;
    if constexpr (GK != GK_POINT) {
      rn[wm] = div_l2(mm, PQ, P.pq_log2);
      const int rem = mm - rn[wm] * PQ;
      rp[wm] = div_l2(rem, P.Q, P.q_log2);
      rq[wm] = rem - rp[wm] * P.Q;
    } else {
      rn[wm] = rp[wm] = rq[wm] = 0;
    }
  }

  f32x4 acc[WM][WN];
#pragma unroll
  for (int wm = 0; wm < WM; ++wm)
#pragma unroll
    for (int j = 0; j < WN; ++j) acc[wm][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Every global load that does not depend on LDS is issued before the LDS staging barrier: the
  // epilogue's streamed operands (residual / skip gradient or the BN input of the ReLU mask, and a
  // second addend: the coarse addend, or the skip gradient of the BN apply) and, for pointwise
  // problems, the first K step's operands.  Each thread owns fixed 16-byte column chunks of rows
  // tid / ncc + k * rpp in the epilogue.
  constexpr int BNc = 16 * WN;
  constexpr int ncc = BNc / VE;       // column chunks per row
  constexpr int rpp = 256 / ncc;      // rows per pass
  constexpr int NCH = BM / rpp;       // chunks per thread
  static_assert(NCH >= 1 && BM % rpp == 0, "epilogue chunk layout");
  const int cc = tid % ncc;
  const int c0 = cc * VE;
  const void* pf = (MODE == MODE_FWD) ? P.res
                   : ((P.flags & EPI_STORE_F32) ? nullptr : (bnmask ? P.zsrc : P.res));
  const void* pf2 = (MODE == MODE_FWD) ? P.ext : (bnapply ? P.res : nullptr);
  uint4 pre[NCH], pre2[NCH];
  auto load_epi = [&]() {
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      const int m = tm * BM + tid / ncc + k * rpp;
      const long o = (long)m * P.ncol + n0 + c0;
      pre[k] = (pf != nullptr && m < P.M) ? *(const uint4*)((const T*)pf + o) : make_uint4(0, 0, 0, 0);
      pre2[k] = (pf2 != nullptr && m < P.M) ? *(const uint4*)((const T*)pf2 + o) : make_uint4(0, 0, 0, 0);
    }
  };
  if constexpr (GK != GK_HALO) load_epi();
  // K steps whose operands are loaded before the barrier: two for the tall 16-column tiles
  // (their 1x1 problems have K = 64 = two steps), one otherwise
  constexpr int ES = (GK == GK_POINT && WM >= 8) ? 2 : 1;
  uint4 a0raw[ES][WM];
  Frag<T> b0[ES][WN];
  if constexpr (GK == GK_POINT) {
#pragma unroll
    for (int es = 0; es < ES; ++es) {
      const int k0 = es * KS + VE * grp;
#pragma unroll
      for (int wm = 0; wm < WM; ++wm)
        a0raw[es][wm] = (rv[wm] && k0 < P.K) ? *(const uint4*)((const T*)P.in + (long)rm[wm] * P.Cg + k0)
                                             : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int j = 0; j < WN; ++j) load_b<T, true>(P, n0 + j * 16 + r16, k0, b0[es][j]);
    }
  }

  if (MODE == MODE_FWD && P.pro != nullptr)
    for (int c = tid; c < P.Cg; c += 256) pro_s[c] = make_float2(P.pro[c], P.pro[P.Cg + c]);
  if (bnmask && tid < 16 * WN) {
    const int col = n0 + tid;
#pragma unroll
    for (int k = 0; k < 4; ++k) bn_s[k][tid] = P.bnst[k * P.ncol + col];
    if (bnapply) {
#pragma unroll
      for (int k = 0; k < 3; ++k) bn_s[4 + k][tid] = P.coef[k * P.ncol + col];
    }
  }
  __syncthreads();

  int kstart = 0;
  if constexpr (GK == GK_POINT) {
    // the early K steps; the BN prologue (scale, shift from LDS) applies now.  Rows past M and
    // columns past K are zeros of the activated operand.
#pragma unroll
    for (int es = 0; es < ES; ++es) {
      const int k0 = es * KS + VE * grp;
      Frag<T> a[WM];
#pragma unroll
      for (int wm = 0; wm < WM; ++wm) {
        if (MODE == MODE_FWD && P.pro != nullptr && rv[wm] && k0 < P.K) {
          Chunk<T> c;
          unpack_chunk<T>(a0raw[es][wm], c);
#pragma unroll
          for (int e = 0; e < VE; ++e) c.v[e] = fmaxf(fmaf(c.v[e], pro_s[k0 + e].x, pro_s[k0 + e].y), 0.0f);
          a[wm].from_chunk(c);
        } else {
          a[wm].from_raw(a0raw[es][wm]);
        }
      }
#pragma unroll
      for (int j = 0; j < WN; ++j)
#pragma unroll
        for (int wm = 0; wm < WM; ++wm) mma(a[wm], b0[es][j], acc[wm][j]);
    }
    kstart = ES * KS;
  }

  if constexpr (GK == GK_HALO) conv_halo<T, MODE, WM, WN>(P, pro_s, (T*)acc_s, tm, n0, acc, load_epi);
  for (int kk = kstart; kk < P.K && GK != GK_HALO; kk += KS) {
    const int k0 = kk + VE * grp;
    Frag<T> a[WM];
#pragma unroll
    for (int wm = 0; wm < WM; ++wm) gather_a<T, MODE, GK>(P, pro_s, rm[wm], rn[wm], rp[wm], rq[wm], rv[wm], k0, a[wm]);
#pragma unroll
    for (int j = 0; j < WN; ++j) {
      Frag<T> b;
      load_b<T, GK != GK_SCALAR>(P, n0 + j * 16 + r16, k0, b);
#pragma unroll
      for (int wm = 0; wm < WM; ++wm) mma(a[wm], b, acc[wm][j]);
    }
  }

  // ---- epilogue: stage the fp32 tile in LDS ----
#pragma unroll
  for (int wm = 0; wm < WM; ++wm)
#pragma unroll
    for (int j = 0; j < WN; ++j) {
      // row / column sub-tile of acc[wm][j]: waves split rows, or (GK_HALO) columns first
      const int rt = (GK == GK_HALO) ? (wave / WN) * (WM * WN) + wm * WN + j : wave * WM + wm;
      const int ct = (GK == GK_HALO) ? wave % WN : j;
#pragma unroll
      for (int i = 0; i < 4; ++i) acc_s[(rt * 16 + grp * 4 + i) * LDA + ct * 16 + r16] = acc[wm][j][i];
    }
  __syncthreads();

  conv_epilogue<T, MODE, BM, BNc, LDA, 64>(P, acc_s, (float*)pro_s, &bn_s[0][0], tm, n0, pre, pre2);
}

// ------------------------------------------------------------------------------------------------
// weight gradient: dW[co][(r,s,c)] = sum_m g[m][co] * act(in)[pixel(m) + tap(r,s)][c]
//
// A workgroup owns a (16 wr) x 64 tile of dW and a range of m (split-K; fp32 partials are summed
// in a fixed order by the column reduce).  Both operands are staged m-major through LDS with
// 16-byte global loads; the MFMA fragments (8 consecutive m per lane) are read column-wise from
// rows padded to 8 bytes past a 16-byte multiple, which keeps the four m-groups of a wave on
// disjoint banks.  wr waves cover the tile's rows; the other 4 / wr wave groups split each LDS
// stage's m-steps and are summed in LDS at the end.  Two register buffers keep the global loads
// of the next two stages in flight while a stage is consumed.
// ------------------------------------------------------------------------------------------------
constexpr int WG_KC = 64;                  // m rows per LDS stage
constexpr int WG_TK = 64;                  // dW columns per workgroup tile

template <typename T>
struct WgCfg {
  static constexpr int VE = St<T>::VE;
  static constexpr int PADE = 8 / sizeof(T);         // 8-byte row padding
  static constexpr int RSA = WG_TK + PADE;            // activation tile row stride (elements)
  static constexpr int AC = WG_KC * WG_TK / VE / 256; // activation chunks per thread per stage
  static constexpr int GC = WG_KC * 64 / VE / 256;    // max output-gradient chunks per thread
};

template <typename T>
__device__ __forceinline__ void lds_store8(T* p, uint4 u) {
  // 16 bytes as two 8-byte stores (rows are 8-byte aligned)
  *(uint2*)p = make_uint2(u.x, u.y);
  *(uint2*)(p + 8 / sizeof(T)) = make_uint2(u.z, u.w);
}

// Column of the activation tile a thread gathers: filter column kidx = (tap, c0), fixed per thread.
struct WgCol {
  int kidx, c0, r, s;
};

__device__ __forceinline__ WgCol wg_col(const WgradProb& P, int kidx) {
  WgCol c;
  c.kidx = kidx;
  const int tap = div_l2(kidx, P.Cg, P.cg_log2);
  c.c0 = kidx - tap * P.Cg;
  tap_rs(tap, P.k, c.r, c.s);
  return c;
}

// One 16-byte activation chunk of row m at the thread's filter column.  VEC: the raw stored values
// (pending = true when the BN prologue still has to be applied, valid = false for padding chunks,
// which are zeros of the activated tensor; both are applied once the load has landed, so that a
// stage's loads stay in flight across the previous stage's MMAs).  Element-wise gather: final
// values (valid = true, pending = false).
template <typename T, bool VEC>
__device__ __forceinline__ uint4 wg_gather(const WgradProb& P, const float2* pro, int m, const WgCol& cl,
                                           int col, bool& valid, bool& pending) {
  constexpr int VE = St<T>::VE;
  const int PQ = P.P * P.Q;
  uint4 zero = make_uint4(0, 0, 0, 0);
  valid = true;
  pending = false;
  if constexpr (VEC) {
    // branch-free: every lane issues its load (padding lanes read the tensor's first chunk and
    // drop it once it has landed: valid = false), so the number of loads in flight is the same on
    // every path
    const bool mv = m < P.M && cl.kidx < P.K;
    const int mm = mv ? m : 0;
    const int n = div_l2(mm, PQ, P.pq_log2);
    const int rem = mm - n * PQ;
    const int p = div_l2(rem, P.Q, P.q_log2);
    const int q = rem - p * P.Q;
    const int ih = p * P.stride + cl.r - P.pad, iw = q * P.stride + cl.s - P.pad;
    const bool v = mv && (unsigned)ih < (unsigned)P.H && (unsigned)iw < (unsigned)P.W;
    const long idx = v ? (((long)n * P.H + ih) * P.W + iw) * P.Cg + cl.c0 : 0;
    valid = v;
    pending = v && P.pro != nullptr;
    return *(const uint4*)((const T*)P.in + idx);
  } else {
    if (m >= P.M || cl.kidx >= P.K) return zero;
    const int n = div_l2(m, PQ, P.pq_log2);
    const int rem = m - n * PQ;
    const int p = div_l2(rem, P.Q, P.q_log2);
    const int q = rem - p * P.Q;
    float v[VE];
#pragma unroll
    for (int e = 0; e < VE; ++e) {
      v[e] = 0.f;
      const int kx = cl.kidx + e;
      if (kx >= P.K) continue;
      const int tap = kx / P.Cg;
      const int ch = kx - tap * P.Cg;
      int r, s;
      tap_rs(tap, P.k, r, s);
      const int ih = p * P.stride + r - P.pad, iw = q * P.stride + s - P.pad;
      if ((unsigned)ih < (unsigned)P.H && (unsigned)iw < (unsigned)P.W) {
        float x = St<T>::ld(P.in, (((long)n * P.H + ih) * P.W + iw) * P.Cg + ch);
        if (P.pro != nullptr) x = fmaxf(fmaf(x, pro[col + e].x, pro[col + e].y), 0.0f);
        v[e] = x;
      }
    }
    uint4 u;
    store_chunk<T>(&u, 0, v);
    return u;
  }
}

// MFMA fragment of 8 (bf16) / 4 (fp32) consecutive m rows at one column of an m-major LDS tile:
// lane (r16, grp) takes rows row0 .. row0 + VE - 1 (row0 includes VE * grp) of column cbase + r16.
// bf16 uses the gfx950 LDS transpose read: within a 16-lane group, lane i receives element i % 4 of
// the 8-byte words supplied by lanes 4e + i / 4 (e = 0..3), so lane j supplies the address of row
// (row0 + j / 4) at column cbase + 4 (j % 4), and a second read covers rows row0 + 4 .. row0 + 7.
typedef short v4s16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s16 lds_v4s16;

template <typename T>
__device__ __forceinline__ void lds_frag(const T* base, int row0, int rs, int cbase, int r16, Frag<T>& f) {
  if constexpr (sizeof(T) == 2) {
    const T* p0 = base + (row0 + (r16 >> 2)) * rs + cbase + 4 * (r16 & 3);
    const v4s16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s16*)p0);
    const v4s16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s16*)(p0 + 4 * rs));
    const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
    f.from_raw(make_uint4(l2.x, l2.y, h2.x, h2.y));
  } else {
    constexpr int VE = St<T>::VE;
    T tmp[VE];
#pragma unroll
    for (int e = 0; e < VE; ++e) tmp[e] = base[(row0 + e) * rs + cbase + r16];
    uint4 u;
    __builtin_memcpy(&u, tmp, 16);
    f.from_raw(u);
  }
}

template <typename T, int GA>
__global__ __launch_bounds__(256) void wgrad_kernel(const WgradLaunch L) {
  using C = WgCfg<T>;
  constexpr int VE = C::VE;
  constexpr int KS = 4 * VE;
  constexpr int LG = WG_KC * (64 + C::PADE);          // output-gradient tile (elements)
  constexpr int LA = WG_KC * C::RSA;                  // activation tile
  constexpr int SMEM = (LG + LA) * (int)sizeof(T) > 16384 ? (LG + LA) * (int)sizeof(T) : 16384;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];   // the two tiles; the final reduce
  __shared__ float2 pro_s[WG_TK];
  T* lg = (T*)smem;
  T* la = lg + LG;

  const int gi = find_group(L);
  const WgradProb& P = L.p[gi];
  const int local = blockIdx.x - P.tile_begin;
  const int tk = local % P.tiles_k;
  const int rest = local / P.tiles_k;
  const int tco = rest % P.tiles_co;
  const int split = rest / P.tiles_co;
  const int TCO = 16 * P.wr;
  const int RSG = TCO + C::PADE;
  const int co0 = tco * TCO;
  const int kk0 = tk * WG_TK;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int r16 = lane & 15, grp = lane >> 4;
  const int sr = wave % P.wr;          // row sub-tile of this wave
  const int ms = 4 / P.wr;             // m-split factor
  const int msi = wave / P.wr;
  const int m_begin = split * P.mchunk;
  const int m_end = min(P.M, m_begin + P.mchunk);

  if (P.pro != nullptr && tid < WG_TK) {
    const int kidx = kk0 + tid;
    const int c = kidx < P.K ? kidx % P.Cg : 0;
    pro_s[tid] = make_float2(P.pro[c], P.pro[P.Cg + c]);
  }
  __syncthreads();

  const int gcpr = TCO / VE;           // output-gradient chunks per row
  const int gchunks = WG_KC * gcpr;
  constexpr int acpr = WG_TK / VE;     // activation chunks per row
  static_assert(256 % acpr == 0, "a thread keeps one activation column");
  const int acol = (tid % acpr) * VE;
  const WgCol wcol = wg_col(P, kk0 + acol);
  // per-thread chunk geometry, fixed over the stages: stage row, element offset in the global
  // tensor relative to the stage's first row, LDS offset (rows past the tile: row = 1 << 29)
  int grow[C::GC], goff[C::GC], gls[C::GC];
#pragma unroll
  for (int i = 0; i < C::GC; ++i) {
    const int idx = tid + i * 256;
    const int row = idx / gcpr, cc = (idx - row * gcpr) * VE;
    const bool in = idx < gchunks;
    grow[i] = in ? row : (1 << 29);
    goff[i] = in ? row * P.Co + co0 + cc : 0;
    gls[i] = in ? row * RSG + cc : -1;
  }
  int arow[C::AC], aoff[C::AC];
  const bool acv = kk0 + acol < P.K;   // the thread's activation column exists
#pragma unroll
  for (int i = 0; i < C::AC; ++i) {
    arow[i] = (tid + i * 256) / acpr;
    aoff[i] = arow[i] * P.Cg + kk0 + acol;   // pointwise gather: row-major [M][Cg] input
  }
  uint4 ga0[C::GC], aa0[C::AC], ga1[C::GC], aa1[C::AC];
  // per stage buffer: bit i of the low byte: ga[i] valid; bit 8 + i: aa[i] valid; bit 16 + i:
  // aa[i] still needs the BN prologue.  Invalid chunks are zeroed when they are written to LDS.
  uint32_t bits0 = 0, bits1 = 0;
  static_assert(C::GC <= 8 && C::AC <= 8, "stage bits");
  const bool has_pro = P.pro != nullptr;

  auto load_stage = [&](uint4 (&ga)[C::GC], uint4 (&aa)[C::AC], uint32_t& bits, int mc) {
    bits = 0;
    const T* gs = (const T*)P.g + (long)mc * P.Co;
#pragma unroll
    for (int i = 0; i < C::GC; ++i) {
      // branch-free like wg_gather: invalid chunks load the tensor's first chunk
      const bool v = mc + grow[i] < m_end;
      ga[i] = *(const uint4*)(v ? gs + goff[i] : (const T*)P.g);
      bits |= (v ? 1u : 0u) << i;
    }
    if constexpr (GA == WG_PW) {
      const T* as = (const T*)P.in + (long)mc * P.Cg;
#pragma unroll
      for (int i = 0; i < C::AC; ++i) {
        const bool v = acv && mc + arow[i] < m_end;
        aa[i] = *(const uint4*)(v ? as + aoff[i] : (const T*)P.in);
        bits |= ((v ? 1u : 0u) << (8 + i)) | ((v && has_pro ? 1u : 0u) << (16 + i));
      }
    } else {
#pragma unroll
      for (int i = 0; i < C::AC; ++i) {
        const int m = mc + arow[i];
        bool valid = true, pend = false;
        aa[i] = wg_gather<T, GA == WG_VEC>(P, pro_s, m < m_end ? m : P.M, wcol, acol, valid, pend);
        bits |= ((valid ? 1u : 0u) << (8 + i)) | ((pend ? 1u : 0u) << (16 + i));
      }
    }
  };
  auto store_stage = [&](const uint4 (&ga)[C::GC], const uint4 (&aa)[C::AC], uint32_t bits) {
#pragma unroll
    for (int i = 0; i < C::GC; ++i)
      if (gls[i] >= 0) lds_store8<T>(lg + gls[i], ((bits >> i) & 1u) ? ga[i] : make_uint4(0, 0, 0, 0));
#pragma unroll
    for (int i = 0; i < C::AC; ++i) {
      uint4 u = ((bits >> (8 + i)) & 1u) ? aa[i] : make_uint4(0, 0, 0, 0);
      if ((bits >> (16 + i)) & 1u) {
        Chunk<T> c;
        unpack_chunk<T>(u, c);
        float v[VE];
#pragma unroll
        for (int e = 0; e < VE; ++e) v[e] = fmaxf(fmaf(c.v[e], pro_s[acol + e].x, pro_s[acol + e].y), 0.0f);
        store_chunk<T>(&u, 0, v);
      }
      lds_store8<T>(la + arow[i] * C::RSA + acol, u);
    }
  };

  f32x4 acc[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // m-step st of stage si goes to wave group (si * steps + st) mod ms
  auto compute = [&](int si) {
#pragma unroll
    for (int st = 0; st < WG_KC / KS; ++st) {
      if (((si * (WG_KC / KS) + st) & (ms - 1)) != msi) continue;
      const int row0 = st * KS + VE * grp;
      Frag<T> a;
      lds_frag<T>(lg, row0, RSG, sr * 16, r16, a);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        Frag<T> b;
        lds_frag<T>(la, row0, C::RSA, j * 16, r16, b);
        mma(a, b, acc[j]);
      }
    }
  };

  // stages alternate between the two register buffers; the loads of stage i + 2 are issued as soon
  // as stage i has been written to LDS.  Every stage's loads are issued, also past m_end (all
  // chunks invalid: zeros), so that the loads in flight are the same on every path and the waits
  // before a stage's LDS stores only cover that stage.
  load_stage(ga0, aa0, bits0, m_begin);
  __builtin_amdgcn_sched_barrier(0);   // keep the two stages' loads in order (the waits count on it)
  load_stage(ga1, aa1, bits1, m_begin + WG_KC);
  for (int mc = m_begin, si = 0; mc < m_end; mc += 2 * WG_KC, si += 2) {
    store_stage(ga0, aa0, bits0);
    __syncthreads();
    load_stage(ga0, aa0, bits0, mc + 2 * WG_KC);
    compute(si);
    __syncthreads();
    store_stage(ga1, aa1, bits1);
    __syncthreads();
    load_stage(ga1, aa1, bits1, mc + 3 * WG_KC);
    compute(si + 1);
    __syncthreads();
  }

  // combine the m-split wave groups (fixed order) and write the partial tile
  float* red = (float*)smem;           // ms x wr x 16 x 64 floats <= 16 KB
  if (ms > 1) {
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        red[((msi * P.wr + sr) * 16 + grp * 4 + i) * 64 + j * 16 + r16] = acc[j][i];
    __syncthreads();
    if (msi == 0) {
      for (int k = 1; k < ms; ++k)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[j][i] += red[((k * P.wr + sr) * 16 + grp * 4 + i) * 64 + j * 16 + r16];
    }
  }
  if (msi != 0) return;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int kidx = kk0 + j * 16 + r16;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int co = co0 + sr * 16 + grp * 4 + i;
      if (co < P.Co && kidx < P.K) P.part[((long)split * P.Co + co) * P.K + kidx] = acc[j][i];
    }
  }
}

// ------------------------------------------------------------------------------------------------
// weight gradient of a 3x3 / stride 1 / pad 1 convolution through an LDS halo tile:
// dW[co][(r,s)][c] = sum_m g[m][co] * act(in)[pixel(m) + (r - 1, s - 1)][c]
//
// A workgroup owns 16 output channels x one 16-channel input block x all 9 taps (9 MFMA column
// tiles) over an m range (split-K in stages of W3_KC rows = whole image rows).  Each stage stages
// the output-gradient rows m-major and the stage's input rows plus a one-pixel halo (BN prologue
// applied when the loads land, zeros for padding) in LDS, once for all taps; the fragments of the
// 8 consecutive m of a lane group are consecutive pixels of one halo row, read with the LDS
// transpose read at the tap's pixel offset.  The four waves split each stage's K steps and are
// summed in LDS in a fixed order at the end.
// ------------------------------------------------------------------------------------------------
template <typename T>
struct W3Cfg {
  static constexpr int VE = St<T>::VE;
  static constexpr int KC = sizeof(T) == 2 ? 256 : 128;   // m rows per stage
  static constexpr int PADE = 8 / sizeof(T);             // 8-byte row padding of the g tile
  static constexpr int RSG = 16 + PADE;
  static constexpr int GC = KC * 16 / VE / 256;          // g chunks per thread
  static constexpr int HC = 4;                           // max halo chunks per thread
  static constexpr int HALO = HC * 256 * VE;             // halo elements
  static constexpr int STAGE_BYTES = (KC * RSG + HALO) * sizeof(T);
  static constexpr int RED_BYTES = 3 * 9 * 256 * 4;      // waves 1..3 x 9 tiles x 16 x 16 floats
  static constexpr int LDS_BYTES = STAGE_BYTES > RED_BYTES ? STAGE_BYTES : RED_BYTES;
};

template <typename T>
__global__ __launch_bounds__(256) void wgrad3_kernel(const WgradLaunch L) {
  using C = W3Cfg<T>;
  constexpr int VE = C::VE;
  constexpr int KS = 4 * VE;
  constexpr int KC = C::KC;
  __shared__ __attribute__((aligned(16))) char smem[C::LDS_BYTES];
  __shared__ float2 pro_s[16];
  T* lg = (T*)smem;
  T* lh = lg + KC * C::RSG;

  const int gi = find_group(L);
  const WgradProb& P = L.p[gi];
  const int local = blockIdx.x - P.tile_begin;
  // a split's tiles (every input block and output-channel tile over the same pixels) read the same
  // gradient and input rows: the first 8 floor(splits / 8) splits grouped by XCD (the XCDs take
  // workgroups round-robin by blockIdx, each with its own L2): local index 8 q + x takes split
  // x + 8 (q / W), tile q % W (W tiles per split); the remaining splits in plain order
  const int W = P.tiles_co * P.tiles_k;
  const int S8 = P.splits & ~7;
  int t, split;
  if (local < S8 * W) {
    const int q = local >> 3;
    split = (local & 7) + 8 * (q / W);
    t = q % W;
  } else {
    const int l2 = local - S8 * W;
    split = S8 + l2 / W;
    t = l2 % W;
  }
  const int tcb = t % P.tiles_k;                    // 16-channel input block
  const int tco = t / P.tiles_k;
  const int co0 = tco * 16, c0 = tcb * 16;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int r16 = lane & 15, grp = lane >> 4;
  const int m_begin = split * P.mchunk;
  const int m_end = min(P.M, m_begin + P.mchunk);
  const int PQ = P.P * P.Q;
  const int QH = P.Q + 2;
  const bool multi = KC > PQ;
  const int R = multi ? P.P : KC / P.Q;             // output rows per image in a stage
  const int RH = R + 2;
  const int nimg = multi ? KC / PQ : 1;
  const int img_px = RH * QH;
  constexpr int cpp = 16 / VE;                      // halo chunks per pixel
  const int hchunks = nimg * img_px * cpp;

  if (P.pro != nullptr && tid < 16) pro_s[tid] = make_float2(P.pro[c0 + tid], P.pro[P.Cg + c0 + tid]);
  __syncthreads();

  uint4 ga[C::GC], ha[C::HC];
  int hoff[C::HC];
  uint32_t hpend = 0;
  const float r_img = 1.0f / img_px, r_qh = 1.0f / QH;

  auto load_stage = [&](int mc) {
#pragma unroll
    for (int i = 0; i < C::GC; ++i) {
      const int idx = tid + i * 256;
      const int row = idx / (16 / VE), cc = (idx % (16 / VE)) * VE;
      const int m = mc + row;
      ga[i] = m < m_end ? *(const uint4*)((const T*)P.g + (long)m * P.Co + co0 + cc) : make_uint4(0, 0, 0, 0);
    }
    const int n_first = div_l2(mc, PQ, P.pq_log2);
    const int p0 = multi ? 0 : div_l2(mc - n_first * PQ, P.Q, P.q_log2);
    hpend = 0;
#pragma unroll
    for (int u = 0; u < C::HC; ++u) {
      const int idx = tid + u * 256;
      const int pix = idx / cpp, ch = idx % cpp;
      int i, rem, y, x;
      if (nimg > 1) divmod_small(pix, img_px, r_img, i, rem);
      else { i = 0; rem = pix; }
      divmod_small(rem, QH, r_qh, y, x);
      const int n = n_first + i, ih = p0 - 1 + y, iw = x - 1;
      const bool ok = idx < hchunks && n < P.B && (unsigned)ih < (unsigned)P.H && (unsigned)iw < (unsigned)P.W;
      hoff[u] = idx < hchunks ? pix * 16 + ch * VE : -1;
      const long gofs = ok ? (((long)n * P.H + ih) * P.W + iw) * P.Cg + c0 + ch * VE : 0;
      ha[u] = ok ? *(const uint4*)((const T*)P.in + gofs) : make_uint4(0, 0, 0, 0);
      hpend |= ((ok && P.pro != nullptr) ? 1u : 0u) << u;
    }
  };
  auto store_stage = [&]() {
#pragma unroll
    for (int i = 0; i < C::GC; ++i) {
      const int idx = tid + i * 256;
      const int row = idx / (16 / VE), cc = (idx % (16 / VE)) * VE;
      lds_store8<T>(lg + row * C::RSG + cc, ga[i]);
    }
#pragma unroll
    for (int u = 0; u < C::HC; ++u) {
      if (hoff[u] < 0) continue;
      uint4 w = ha[u];
      if ((hpend >> u) & 1u) {
        const int cb = hoff[u] & 15;            // channel offset within the block
        Chunk<T> c;
        unpack_chunk<T>(w, c);
        float v[VE];
#pragma unroll
        for (int e = 0; e < VE; ++e) v[e] = fmaxf(fmaf(c.v[e], pro_s[cb + e].x, pro_s[cb + e].y), 0.0f);
        store_chunk<T>(&w, 0, v);
      }
      *(uint4*)(lh + hoff[u]) = w;
    }
  };

  f32x4 acc[9];
#pragma unroll
  for (int t = 0; t < 9; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (m_begin < m_end) load_stage(m_begin);
  for (int mc = m_begin; mc < m_end; mc += KC) {
    store_stage();
    __syncthreads();
    if (mc + KC < m_end) load_stage(mc + KC);
    for (int st = wave; st < KC / KS; st += 4) {
      const int row0 = st * KS + VE * grp;        // first of the lane group's VE rows of the stage
      Frag<T> a;
      lds_frag<T>(lg, row0, C::RSG, 0, r16, a);
      const int i = multi ? div_l2(row0, PQ, P.pq_log2) : 0;
      const int rem = row0 - i * PQ;
      const int pl = div_l2(rem, P.Q, P.q_log2);
      const int ql = rem - pl * P.Q;
      const int pix0 = (i * RH + pl) * QH + ql;   // halo pixel of tap (0, 0)
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const int r = t / 3, s = t - 3 * (t / 3);
        Frag<T> b;
        lds_frag<T>(lh, pix0 + r * QH + s, 16, 0, r16, b);
        mma(a, b, acc[t]);
      }
    }
    __syncthreads();
  }

  // sum the four waves' K-step shares in wave order, then write the 16 x 144 partial tile
  float* red = (float*)smem;
  if (wave > 0) {
#pragma unroll
    for (int t = 0; t < 9; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[((wave - 1) * 9 + t) * 256 + (grp * 4 + i) * 16 + r16] = acc[t][i];
  }
  __syncthreads();
  if (wave != 0) return;
  for (int w = 0; w < 3; ++w)
#pragma unroll
    for (int t = 0; t < 9; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) acc[t][i] += red[(w * 9 + t) * 256 + (grp * 4 + i) * 16 + r16];
#pragma unroll
  for (int t = 0; t < 9; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int co = co0 + grp * 4 + i;
      P.part[((long)split * P.Co + co) * P.K + t * P.Cg + c0 + r16] = acc[t][i];
    }
}

// ------------------------------------------------------------------------------------------------
// BN backward sums of a 1x1 convolution's input BN without forming its data gradient in HBM:
// per row m and column c, v = sum_o g[m][o] W[o][c] (transposed filter wmat[c][o]), dbn =
// rnd(v * [ReLU(BN(z)) > 0]), sums of dbn and dbn * xhat.  A workgroup owns 64 columns and
// P.wm * BNSUM_TR rows and streams them in tiles of BNSUM_TR rows: g (contiguous, BNSUM_TR * K
// elements) and z (BNSUM_TR rows of 64 columns) go through LDS with whole-workgroup 16-byte loads,
// the next tile's loads in flight while the current one is computed.  Wave w owns columns
// [16 w, 16 w + 16); its MFMA takes the filter as the row operand and 16 gradient rows as the
// column operand, so a lane's results are four consecutive columns of one row.  One partial row
// [tiles_m][ncol][2] per workgroup; nothing else is stored.  EPI_PW_WGRAD: the same tiles also
// give the convolution's weight gradient dW[o][c] = sum_m g[m][o] ReLU(BN(z))[m][c]: wave w forms
// the columns c0 + 16 w .. c0 + 16 w + 15 of every 16-row block of o (the gradient tile read
// column-wise as the row operand, the activated BN input as the column operand) and writes them to
// the split-K partial row tm of out32 [tiles_m][K][ncol].
// ------------------------------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(256) void bnsum_kernel(const ConvLaunch L) {
  constexpr int VE = St<T>::VE;
  constexpr int KS = 4 * VE;
  constexpr int NOS = BNSUM_MAXK / KS;                // K steps over the gradient's channels
  constexpr int TR = BNSUM_TR;
  constexpr int ST = 64 + VE;                         // LDS row stride of both tiles (elements)
  constexpr int NLD = TR * 64 / VE / 256;             // 16-byte loads per thread for a full tile
  __shared__ __attribute__((aligned(16))) T gs[TR * ST];
  __shared__ __attribute__((aligned(16))) T zs[TR * ST];

  const int gi = find_group(L);
  const ConvProb& P = L.p[gi];
  const int local = blockIdx.x - P.tile_begin;
  const int tm = local / P.tiles_n;
  const int tn = local - tm * P.tiles_n;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int r16 = lane & 15, grp = lane >> 4;
  const int K = P.K, ncol = P.ncol;
  const int c0 = tn * 64;
  const int ncl = min(64, ncol - c0);                 // columns of this tile (16, 32, 48 or 64)
  const int m_begin = tm * (P.wm * TR);
  const int m_end = min(P.M, m_begin + P.wm * TR);
  const int gch = K / VE;                             // 16-byte chunks per gradient row
  const T* __restrict__ g = (const T*)P.in;
  const T* __restrict__ z = (const T*)P.zsrc;
  const bool active = wave * 16 < ncl;                // the wave has columns

  // filter fragments (column c0 + 16 wave + r16, gradient channels os * KS + VE * grp ..) and the
  // BN parameters of the lane's result columns c0 + 16 wave + 4 grp + i
  Frag<T> wf[NOS];
  float mu[4], is[4], sc[4], sh[4];
  {
    const int c = wave * 16 + r16;
#pragma unroll
    for (int os = 0; os < NOS; ++os) {
      const int o0 = os * KS + VE * grp;
      if (o0 < K && c < ncl) wf[os].from_raw(*(const uint4*)((const T*)P.wmat + (long)(c0 + c) * K + o0));
      else wf[os].zero();
    }
    const int cl = wave * 16 + grp * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool cv = cl + i < ncl;
      mu[i] = cv ? P.bnst[c0 + cl + i] : 0.f;
      is[i] = cv ? P.bnst[ncol + c0 + cl + i] : 0.f;
      sc[i] = cv ? P.bnst[2 * ncol + c0 + cl + i] : 0.f;
      sh[i] = cv ? P.bnst[3 * ncol + c0 + cl + i] : 0.f;
    }
  }

  // fused weight gradient: BN scale / shift of the lane's activation column c0 + 16 wave + r16
  constexpr int NOB = BNSUM_MAXK / 16;                // 16-row blocks of o
  const bool wgr = (P.flags & EPI_PW_WGRAD) != 0 && active;
  f32x4 dw[NOB];
#pragma unroll
  for (int ob = 0; ob < NOB; ++ob) dw[ob] = f32x4{0.f, 0.f, 0.f, 0.f};
  float wsc = 0.f, wsh = 0.f;
  if (wgr && wave * 16 + r16 < ncl) {
    wsc = P.bnst[2 * ncol + c0 + wave * 16 + r16];
    wsh = P.bnst[3 * ncol + c0 + wave * 16 + r16];
  }

  // chunk u of the g tile is row u / gch, channels VE * (u % gch); chunk u of the z tile is row
  // u / (64 / VE), columns VE * (u % (64 / VE))
  uint4 gr[NLD], zr[NLD];
  auto fetch = [&](int mt) {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int u = i * 256 + tid;
      const int row = u / gch;
      gr[i] = (row < TR && mt + row < m_end) ? *(const uint4*)(g + (long)mt * K + (long)u * VE)
                                              : make_uint4(0, 0, 0, 0);
      const int zrow = u / (64 / VE), zc = (u % (64 / VE)) * VE;
      zr[i] = (mt + zrow < m_end && zc < ncl) ? *(const uint4*)(z + (long)(mt + zrow) * ncol + c0 + zc)
                                               : make_uint4(0, 0, 0, 0);
    }
  };

  float s1[4] = {0.f, 0.f, 0.f, 0.f}, s2[4] = {0.f, 0.f, 0.f, 0.f};
  fetch(m_begin);
  for (int mt = m_begin; mt < m_end; mt += TR) {
#pragma unroll
    for (int i = 0; i < NLD; ++i) {
      const int u = i * 256 + tid;
      const int row = u / gch;
      if (row < TR) *(uint4*)(gs + row * ST + (u - row * gch) * VE) = gr[i];
      const int zrow = u / (64 / VE);
      *(uint4*)(zs + zrow * ST + (u % (64 / VE)) * VE) = zr[i];
    }
    __syncthreads();
    if (mt + TR < m_end) fetch(mt + TR);
    if (active) {
#pragma unroll
      for (int sub = 0; sub < TR / 16; ++sub) {
        const int row = sub * 16 + r16;
        f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int os = 0; os < NOS; ++os) {
          const int o0 = os * KS + VE * grp;
          if (os * KS < K) {
            Frag<T> gf;
            if (o0 < K) gf.from_raw(*(const uint4*)(gs + row * ST + o0));
            else gf.zero();
            mma(wf[os], gf, v);
          }
        }
        float zv[4];
        const int cl = wave * 16 + grp * 4;
        if constexpr (sizeof(T) == 2) {
          const uint2 u = *(const uint2*)(zs + row * ST + cl);
          zv[0] = __uint_as_float(u.x << 16);
          zv[1] = __uint_as_float(u.x & 0xffff0000u);
          zv[2] = __uint_as_float(u.y << 16);
          zv[3] = __uint_as_float(u.y & 0xffff0000u);
        } else {
          const float4 u = *(const float4*)(zs + row * ST + cl);
          zv[0] = u.x; zv[1] = u.y; zv[2] = u.z; zv[3] = u.w;
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float d = fmaf(zv[i], sc[i], sh[i]) > 0.f ? v[i] : 0.f;
          const float dr = St<T>::rnd(d);
          s1[i] += dr;
          s2[i] += dr * ((zv[i] - mu[i]) * is[i]);
        }
      }
    }
    if (wgr) {
      // rows past m_end are zeros of g in the tile, so they add nothing
#pragma unroll
      for (int ms = 0; ms < TR / KS; ++ms) {
        const int row0 = ms * KS + VE * grp;
        Frag<T> af;
        lds_frag<T>(zs, row0, ST, wave * 16, r16, af);
#pragma unroll
        for (int e = 0; e < (int)(sizeof(af.v) / sizeof(af.v[0])); ++e) {
          const float a = fmaxf(fmaf((float)af.v[e], wsc, wsh), 0.0f);
          if constexpr (sizeof(T) == 2) af.v[e] = (__bf16)a;
          else af.v[e] = a;
        }
#pragma unroll
        for (int ob = 0; ob < NOB; ++ob) {
          if (ob * 16 < K) {
            Frag<T> gf;
            lds_frag<T>(gs, row0, ST, ob * 16, r16, gf);
            mma(gf, af, dw[ob]);
          }
        }
      }
    }
    __syncthreads();
  }
  if (wgr && wave * 16 + r16 < ncl) {
    // lane (r16, grp) holds rows o = 16 ob + 4 grp + i of column c0 + 16 wave + r16
    float* dst = P.out32 + (long)tm * K * ncol + c0 + wave * 16 + r16;
#pragma unroll
    for (int ob = 0; ob < NOB; ++ob)
      if (ob * 16 < K)
#pragma unroll
        for (int i = 0; i < 4; ++i) dst[(long)(ob * 16 + 4 * grp + i) * ncol] = dw[ob][i];
  }
  // sum over the 16 rows of a lane group (lanes r16); lane r16 == 0 holds four columns
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      s1[i] += __shfl_xor(s1[i], o, 64);
      s2[i] += __shfl_xor(s2[i], o, 64);
    }
  if (active && r16 == 0) {
    const int cl = wave * 16 + grp * 4;
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (cl + i < ncl) ((float2*)P.part)[(long)tm * ncol + c0 + cl + i] = make_float2(s1[i], s2[i]);
  }
}

// ------------------------------------------------------------------------------------------------
// Streaming pointwise convolution (1x1, stride 1, pad 0, K <= MAXK), used for narrow problems
// (16-column tiles), where it keeps more loads in flight than the 512-row conv tile:
//   FWD: out[m][c] = sum_k act(x[m][k]) W[c][k], act = ReLU(x * scale + shift) (P.pro) or identity;
//        stored rounded; EPI_STATS: column sums of the stored value and of its square -> part.
//   BWD (EPI_BN_MASK): v[m][c] = sum_o g[m][o] Wt[c][o]; dbn = rnd(v * [ReLU(BN(z)) > 0]), stored
//        unless EPI_NO_STORE; sums of dbn and dbn * xhat -> part.
// A workgroup owns 16 CW columns and P.wm tiles of PW_TR rows, streamed one tile after the other: the input rows
// (contiguous, PW_TR * K elements; the FWD prologue applied as they are written) and for BWD the BN
// input go through LDS with whole-workgroup 16-byte loads, the next tile's loads in flight while the
// current one is computed.  Waves: CW columns of 16 times 4 / CW row groups.  A wave's MFMA takes
// its 16 filter rows as the row operand and 16 input rows as the column operand, so a lane's
// results are four consecutive columns of one row.  One partial row [tiles_m][ncol][2] per workgroup.
// BWD + EPI_PW_WGRAD (CW = 1): the same LDS tiles also give the convolution's weight gradient
// dW[o][c] = sum_m g[m][o] ReLU(BN(z))[m][c]: wave w accumulates rows o = 16 w .. 16 w + 15 (the
// gradient tile read column-wise as the row operand, the activated BN input as the column
// operand) and writes them to the split-K partial row tm of out32 [tiles_m][K][ncol].
// ------------------------------------------------------------------------------------------------
template <typename T, int MODE, int CW, int MAXK>
__global__ __launch_bounds__(256) void pw_kernel(const ConvLaunch L) {
  constexpr int VE = St<T>::VE;
  constexpr int KS = 4 * VE;
  constexpr int NOS = MAXK / KS;                      // K steps
  constexpr int TR = PW_TR;
  constexpr int NC = 16 * CW;                         // columns of the workgroup tile
  constexpr int WR = 4 / CW;                          // wave row groups
  constexpr int SZ = NC + VE;                         // LDS row stride of the BN-input tile
  constexpr int NLA = TR * MAXK / VE / 256;           // 16-byte input loads per thread
  constexpr int NLZ = (TR * NC / VE + 255) / 256;     // 16-byte BN-input loads per thread
  __shared__ __attribute__((aligned(16))) T xs[TR * (MAXK + VE)];
  __shared__ __attribute__((aligned(16))) T zs[MODE == MODE_BWD ? TR * SZ : 8];
  __shared__ float2 pro_s[MODE == MODE_FWD ? MAXK : 1];
  __shared__ float2 red[WR][NC];
  __shared__ float piv[MODE == MODE_FWD ? NC : 1];
  __shared__ float pivp[MODE == MODE_FWD ? 256 : 1];   // pivot dot-product partials [256 / NC][NC]

  const int gi = find_group(L);
  const ConvProb& P = L.p[gi];
  const int local = blockIdx.x - P.tile_begin;
  const int tm = local / P.tiles_n;
  const int tn = local - tm * P.tiles_n;
  const int tid = threadIdx.x;
  const int wave = tid >> 6, lane = tid & 63;
  const int r16 = lane & 15, grp = lane >> 4;
  const int wr = wave / CW, wc = wave % CW;
  const int K = P.K, ncol = P.ncol;
  const int c0 = tn * NC;
  const int ncl = min(NC, ncol - c0);                 // columns of this tile (a multiple of 16)
  const int m_begin = tm * (P.wm * TR);               // P.wm tiles of TR rows per workgroup
  const int m_end = min(P.M, m_begin + P.wm * TR);
  const int gch = K / VE;                             // 16-byte chunks per input row
  const int SA = K + VE;                              // LDS row stride of the input tile (elements)
  const T* __restrict__ xin = (const T*)P.in;
  const T* __restrict__ z = (const T*)P.zsrc;
  const bool active = wc * 16 < ncl;                  // the wave's 16 columns exist
  const bool pro = MODE == MODE_FWD && P.pro != nullptr;
  const bool stats = MODE == MODE_FWD ? (P.flags & EPI_STATS) != 0 : true;
  const bool store = MODE == MODE_FWD || !(P.flags & EPI_NO_STORE);

  if constexpr (MODE == MODE_FWD) {
    if (pro)
      for (int k = tid; k < K; k += 256) pro_s[k] = make_float2(P.pro[k], P.pro[P.Cg + k]);
  }
  // filter fragments (column c0 + 16 wc + r16, channels os * KS + VE * grp ..) and the BN
  // parameters of the lane's result columns c0 + 16 wc + 4 grp + i
  Frag<T> wf[NOS];
  const int cl = wc * 16 + grp * 4;
  float mu[4], is[4], sc[4], sh[4];
  {
    const int c = wc * 16 + r16;
#pragma unroll
    for (int os = 0; os < NOS; ++os) {
      const int o0 = os * KS + VE * grp;
      if (o0 < K && c < ncl) wf[os].from_raw(*(const uint4*)((const T*)P.wmat + (long)(c0 + c) * K + o0));
      else wf[os].zero();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool cv = MODE == MODE_BWD && cl + i < ncl;
      mu[i] = cv ? P.bnst[c0 + cl + i] : 0.f;
      is[i] = cv ? P.bnst[ncol + c0 + cl + i] : 0.f;
      sc[i] = cv ? P.bnst[2 * ncol + c0 + cl + i] : 0.f;
      sh[i] = cv ? P.bnst[3 * ncol + c0 + cl + i] : 0.f;
    }
  }

  // fused weight gradient: BN scale / shift of the lane's activation column c0 + r16
  const bool wgr = MODE == MODE_BWD && CW == 1 && (P.flags & EPI_PW_WGRAD) != 0;
  const bool wact = wgr && 16 * wave < K;
  f32x4 dw = f32x4{0.f, 0.f, 0.f, 0.f};
  float wsc = 0.f, wsh = 0.f;
  if (wgr && r16 < ncl) {
    wsc = P.bnst[2 * ncol + c0 + r16];
    wsh = P.bnst[3 * ncol + c0 + r16];
  }

  // chunk u of the input tile is row u / gch, channels VE * (u % gch); chunk u of the BN-input tile
  // is row u / (NC / VE), columns VE * (u % (NC / VE))
  uint4 xr[NLA], zr[NLZ];
  auto fetch = [&](int mt) {
#pragma unroll
    for (int i = 0; i < NLA; ++i) {
      const int u = i * 256 + tid;
      const int row = u / gch;
      xr[i] = (row < TR && mt + row < m_end) ? *(const uint4*)(xin + (long)mt * K + (long)u * VE)
                                              : make_uint4(0, 0, 0, 0);
    }
    if constexpr (MODE == MODE_BWD) {
#pragma unroll
      for (int i = 0; i < NLZ; ++i) {
        const int u = i * 256 + tid;
        const int zrow = u / (NC / VE), zc = (u % (NC / VE)) * VE;
        zr[i] = (zrow < TR && mt + zrow < m_end && zc < ncl)
                    ? *(const uint4*)(z + (long)(mt + zrow) * ncol + c0 + zc) : make_uint4(0, 0, 0, 0);
      }
    }
  };

  float s1[4] = {0.f, 0.f, 0.f, 0.f}, s2[4] = {0.f, 0.f, 0.f, 0.f};
  fetch(m_begin);
  // Forward BN statistics are summed about a per-workgroup pivot, the first row's output (an fp32
  // dot product here, its K terms split over 256 / NC threads per column; its loads overlap the
  // first tile's), so that they do not cancel when a channel's mean is large against its spread
  if (MODE == MODE_FWD && stats && sizeof(pivp) == 256 * sizeof(float)) {
    constexpr int NQ = 256 / NC;
    const int pc = tid % NC, pq = tid / NC;
    const int kq = (K + NQ - 1) / NQ;
    float a = 0.f;
    if (pc < ncl)
      for (int k = pq * kq; k < min(K, (pq + 1) * kq); ++k) {
        float x = St<T>::ld(xin, (long)m_begin * K + k);
        if (pro) x = fmaxf(fmaf(x, P.pro[k], P.pro[P.Cg + k]), 0.0f);
        a = fmaf(x, St<T>::ld(P.wmat, (long)(c0 + pc) * K + k), a);
      }
    pivp[tid] = a;
  }
  __syncthreads();                                    // pro_s, pivp
  if (MODE == MODE_FWD && stats && tid < ncl && sizeof(piv) == NC * sizeof(float)) {   // read after the first tile's barrier
    float v = 0.f;
    for (int q = 0; q < 256 / NC; ++q) v += pivp[q * NC + tid];
    piv[tid] = St<T>::rnd(v);
  }
  for (int mt = m_begin; mt < m_end; mt += TR) {
#pragma unroll
    for (int i = 0; i < NLA; ++i) {
      const int u = i * 256 + tid;
      const int row = u / gch;
      if (row >= TR) continue;
      const int ch = (u - row * gch) * VE;
      uint4 w = xr[i];
      if (pro && mt + row < m_end) {
        Chunk<T> cx;
        unpack_chunk<T>(w, cx);
        float f[VE];
#pragma unroll
        for (int e = 0; e < VE; ++e) f[e] = fmaxf(fmaf(cx.v[e], pro_s[ch + e].x, pro_s[ch + e].y), 0.0f);
        store_chunk<T>(&w, 0, f);
      }
      *(uint4*)(xs + row * SA + ch) = w;
    }
    if constexpr (MODE == MODE_BWD) {
#pragma unroll
      for (int i = 0; i < NLZ; ++i) {
        const int u = i * 256 + tid;
        const int zrow = u / (NC / VE);
        if (zrow < TR) *(uint4*)(zs + zrow * SZ + (u % (NC / VE)) * VE) = zr[i];
      }
    }
    __syncthreads();
    if (mt + TR < m_end) fetch(mt + TR);
    if (active) {
#pragma unroll
      for (int b = 0; b < CW; ++b) {
        const int row = (wr * CW + b) * 16 + r16;
        const int m = mt + row;
        f32x4 v = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int os = 0; os < NOS; ++os) {
          if (os * KS < K) {
            const int o0 = os * KS + VE * grp;
            Frag<T> xf;
            if (o0 < K) xf.from_raw(*(const uint4*)(xs + row * SA + o0));
            else xf.zero();
            mma(wf[os], xf, v);
          }
        }
        const bool mv = m < m_end;
        float o[4];
        if constexpr (MODE == MODE_FWD) {
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            o[i] = v[i];
            const float d = St<T>::rnd(v[i]) - (stats ? piv[cl + i] : 0.f);
            if (stats && mv) {
              s1[i] += d;
              s2[i] += d * d;
            }
          }
        } else {
          float zv[4];
          if constexpr (sizeof(T) == 2) {
            const uint2 u = *(const uint2*)(zs + row * SZ + cl);
            zv[0] = __uint_as_float(u.x << 16);
            zv[1] = __uint_as_float(u.x & 0xffff0000u);
            zv[2] = __uint_as_float(u.y << 16);
            zv[3] = __uint_as_float(u.y & 0xffff0000u);
          } else {
            const float4 u = *(const float4*)(zs + row * SZ + cl);
            zv[0] = u.x; zv[1] = u.y; zv[2] = u.z; zv[3] = u.w;
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float d = fmaf(zv[i], sc[i], sh[i]) > 0.f ? v[i] : 0.f;
            const float dr = St<T>::rnd(d);
            o[i] = d;
            s1[i] += dr;
            s2[i] += dr * ((zv[i] - mu[i]) * is[i]);
          }
        }
        if (store && mv) {
          T* dst = (T*)P.out + (long)m * ncol + c0 + cl;
          if constexpr (sizeof(T) == 2) {
            *(uint2*)dst = make_uint2((uint32_t)f2bf(o[0]) | ((uint32_t)f2bf(o[1]) << 16),
                                      (uint32_t)f2bf(o[2]) | ((uint32_t)f2bf(o[3]) << 16));
          } else {
            *(float4*)dst = make_float4(o[0], o[1], o[2], o[3]);
          }
        }
      }
    }
    if constexpr (MODE == MODE_BWD && CW == 1) {
      if (wact) {
        // rows past m_end are zeros of g in the tile, so they add nothing
#pragma unroll
        for (int ms = 0; ms < TR / KS; ++ms) {
          const int row0 = ms * KS + VE * grp;
          Frag<T> gf, af;
          lds_frag<T>(xs, row0, SA, 16 * wave, r16, gf);
          lds_frag<T>(zs, row0, SZ, 0, r16, af);
#pragma unroll
          for (int e = 0; e < (int)(sizeof(af.v) / sizeof(af.v[0])); ++e) {
            const float a = fmaxf(fmaf((float)af.v[e], wsc, wsh), 0.0f);
            if constexpr (sizeof(T) == 2) af.v[e] = (__bf16)a;
            else af.v[e] = a;
          }
          mma(gf, af, dw);
        }
      }
    }
    __syncthreads();
  }
  if (wact && r16 < ncl) {
    // lane (r16, grp) holds rows o = 16 wave + 4 grp + i of column c0 + r16
    float* dst = P.out32 + (long)tm * K * ncol + c0 + r16;
#pragma unroll
    for (int i = 0; i < 4; ++i) dst[(long)(16 * wave + 4 * grp + i) * ncol] = dw[i];
  }
  if (!stats) return;
  // sum over the 16 rows of a lane group (lanes r16), then over the wave row groups in order
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      s1[i] += __shfl_xor(s1[i], o, 64);
      s2[i] += __shfl_xor(s2[i], o, 64);
    }
  if (active && r16 == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wr][cl + i] = make_float2(s1[i], s2[i]);
  }
  __syncthreads();
  if (tid < ncl) {
    float a = 0.f, b = 0.f;
#pragma unroll
    for (int w = 0; w < WR; ++w) {
      a += red[w][tid].x;
      b += red[w][tid].y;
    }
    if (MODE == MODE_FWD) {
      // the workgroup's mean and sum of squared deviations from its pivoted sums
      const float am = a / (float)(m_end - m_begin);
      st_coherent((float2*)P.part + (long)tm * ncol + c0 + tid, make_float2(piv[tid] + am, fmaxf(b - a * am, 0.f)));
    } else {
      ((float2*)P.part)[(long)tm * ncol + c0 + tid] = make_float2(a, b);
    }
  }
  if (MODE == MODE_FWD && (P.flags & EPI_BN_FUSE))
    bn_fwd_fuse((float2*)P.part, P.tiles_m, P.wm * TR, (long)P.M, ncol, P.bn_gamma, P.bn_stats, P.bn_cnt, tm, tn, c0,
                ncl, (double*)xs);
}

// ------------------------------------------------------------------------------------------------
// launchers
// ------------------------------------------------------------------------------------------------

template <typename T, int MODE, int WM, int WN>
static void launch_conv_v(const ConvLaunch& L, int tiles, int gk, hipStream_t s) {
  if (gk == GK_POINT)
    hipLaunchKernelGGL((conv_kernel<T, MODE, GK_POINT, WM, WN>), dim3(tiles), dim3(256), 0, s, L);
  else if (gk == GK_VEC)
    hipLaunchKernelGGL((conv_kernel<T, MODE, GK_VEC, WM, WN>), dim3(tiles), dim3(256), 0, s, L);
  else if (gk == GK_HALO)
    hipLaunchKernelGGL((conv_kernel<T, MODE, GK_HALO, WM, WN>), dim3(tiles), dim3(256), 0, s, L);
  else
    hipLaunchKernelGGL((conv_kernel<T, MODE, GK_SCALAR, WM, WN>), dim3(tiles), dim3(256), 0, s, L);
}

// tile variants: (wn, wm) = (1, 8), (2, 4), (4, 2) tall; (1, 2), (2, 1), (4, 1) short
template <typename T, int MODE>
static int launch_conv_m(const ConvLaunch& L, int tiles, int gk, int wn, int wm, hipStream_t s) {
  if (wn == 1 && wm == 8) launch_conv_v<T, MODE, 8, 1>(L, tiles, gk, s);
  else if (wn == 2 && wm == 4) launch_conv_v<T, MODE, 4, 2>(L, tiles, gk, s);
  else if (wn == 4 && wm == 2) launch_conv_v<T, MODE, 2, 4>(L, tiles, gk, s);
  else if (wn == 1 && wm == 2) launch_conv_v<T, MODE, 2, 1>(L, tiles, gk, s);
  else if (wn == 2 && wm == 1) launch_conv_v<T, MODE, 1, 2>(L, tiles, gk, s);
  else if (wn == 4 && wm == 1) launch_conv_v<T, MODE, 1, 4>(L, tiles, gk, s);
  else return (int)hipErrorInvalidValue;
  return 0;
}

int launch_conv(const ConvLaunch& L, int tiles, int dtype, int mode, int gk, int wn, int wm, hipStream_t s) {
  int e;
  if (dtype == 1)
    e = mode == MODE_FWD ? launch_conv_m<uint16_t, MODE_FWD>(L, tiles, gk, wn, wm, s)
                         : launch_conv_m<uint16_t, MODE_BWD>(L, tiles, gk, wn, wm, s);
  else
    e = mode == MODE_FWD ? launch_conv_m<float, MODE_FWD>(L, tiles, gk, wn, wm, s)
                         : launch_conv_m<float, MODE_BWD>(L, tiles, gk, wn, wm, s);
  return e ? e : (int)hipGetLastError();
}

int launch_pw(const ConvLaunch& L, int tiles, int dtype, int mode, hipStream_t s) {
  if (dtype == 1) {
    if (mode == MODE_FWD) hipLaunchKernelGGL((pw_kernel<uint16_t, MODE_FWD, 1, PW_MAXK>), dim3(tiles), dim3(256), 0, s, L);
    else hipLaunchKernelGGL((pw_kernel<uint16_t, MODE_BWD, 1, PW_MAXK>), dim3(tiles), dim3(256), 0, s, L);
  } else {
    if (mode == MODE_FWD) hipLaunchKernelGGL((pw_kernel<float, MODE_FWD, 1, PW_MAXK>), dim3(tiles), dim3(256), 0, s, L);
    else hipLaunchKernelGGL((pw_kernel<float, MODE_BWD, 1, PW_MAXK>), dim3(tiles), dim3(256), 0, s, L);
  }
  return (int)hipGetLastError();
}

int launch_bnsum(const ConvLaunch& L, int tiles, int dtype, hipStream_t s) {
  if (dtype == 1) hipLaunchKernelGGL((bnsum_kernel<uint16_t>), dim3(tiles), dim3(256), 0, s, L);
  else hipLaunchKernelGGL((bnsum_kernel<float>), dim3(tiles), dim3(256), 0, s, L);
  return (int)hipGetLastError();
}

int launch_wgrad3(const WgradLaunch& L, int tiles, int dtype, hipStream_t s) {
  if (dtype == 1)
    hipLaunchKernelGGL((wgrad3_kernel<uint16_t>), dim3(tiles), dim3(256), 0, s, L);
  else
    hipLaunchKernelGGL((wgrad3_kernel<float>), dim3(tiles), dim3(256), 0, s, L);
  return (int)hipGetLastError();
}

template <typename T>
static void launch_wgrad_t(const WgradLaunch& L, int tiles, int gather, hipStream_t s) {
  if (gather == WG_PW) hipLaunchKernelGGL((wgrad_kernel<T, WG_PW>), dim3(tiles), dim3(256), 0, s, L);
  else if (gather == WG_VEC) hipLaunchKernelGGL((wgrad_kernel<T, WG_VEC>), dim3(tiles), dim3(256), 0, s, L);
  else hipLaunchKernelGGL((wgrad_kernel<T, WG_GEN>), dim3(tiles), dim3(256), 0, s, L);
}

int launch_wgrad(const WgradLaunch& L, int tiles, int dtype, int gather, hipStream_t s) {
  if (dtype == 1) {
    launch_wgrad_t<uint16_t>(L, tiles, gather, s);
  } else {
    launch_wgrad_t<float>(L, tiles, gather, s);
  }
  return (int)hipGetLastError();
}


}  // namespace pnn
