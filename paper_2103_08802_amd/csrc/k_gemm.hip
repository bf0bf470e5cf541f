// Implicit-GEMM kernel for the wide 3x3 convolutions (forward and data gradient) of the parareal
// VGG sub-networks (Table vgg: 128-512 channels, K = 9 C_in = 1152-4608 per output) for gfx950,
// where the contraction, not HBM, bounds the layer: bf16 v_mfma_f32_32x32x16_bf16 with fp32
// accumulation, operands staged through LDS.
//
// A workgroup of four waves owns a 128 x 128 output tile (rows = output pixels, columns = output
// channels); each wave a 64 x 64 quarter as 2 x 2 MFMA tiles of 32 x 32.  K runs in steps of GEMM_BK
// (one filter tap and GEMM_BK channels per step, C_in being a multiple of it): the step's A rows (the
// 128 output pixels' input pixels at the tap, BN prologue applied on the way into LDS, zeros for
// padding) and B rows (128 filter rows) are loaded with 16-byte vector loads two steps ahead of
// their use, written to one of two LDS stages, and read back as MFMA fragments from rows padded by
// 16 bytes (conflict-free 16-byte fragment reads).  The fp32 tile is then staged in LDS and the
// convolution epilogue shared with the other conv kernels does residual, BN-mask / BN-apply forms,
// stores and per-tile BN partials (128-row tiles, the same partial rows as the other kernels).
// Problems with few tiles split K over several workgroups per tile (fp32 partial tiles, summed in
// split order by a second pass that then runs the epilogue).
#include "device_common.h"
#include "pnn_internal.h"
#include "conv_epilogue.h"

namespace pnn {

namespace {

constexpr int GM = GEMM_BM, GN = GEMM_BN, GKS = GEMM_BK;   // tile rows, columns; K per step
constexpr int GAS = GKS + 8;                          // LDS row stride of an operand tile (bf16)
constexpr int GLDA = GN + 4;                          // row stride of the staged fp32 tile
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int GCH = GKS / 8;                          // 16-byte chunks per operand row and step
constexpr int GLR = 256 / GCH;                        // rows per loader pass
constexpr int GLP = GM / GLR;                         // loader passes (chunks per thread and operand)
static_assert(GM == 128 && GN == 128 && GM % GLR == 0, "gemm tile: four waves of 64 x 64");

// the tile geometry of a column-tile width TN (128: four waves of 64 x 64; 64: four waves of 32 x 64)
template <int TN>
struct GemmTile {
  static constexpr int OPS = GM * GAS + TN * GAS;     // bf16 elements of one stage (A then B)
  static constexpr int LDA = TN + 4;                  // row stride of the staged fp32 tile
  static constexpr int SMEM = 2 * OPS * 2 > GM * LDA * 4 ? 2 * OPS * 2 : GM * LDA * 4;   // bytes
  static constexpr int LPB = TN / GLR;                // loader passes of the filter rows
  static constexpr int WROWS = TN == 128 ? 64 : 32;   // rows per wave
  static constexpr int MI = WROWS / 32;               // 32-row MFMA blocks per wave
  static_assert(TN == 128 || TN == 64, "column tile");
};

}  // namespace

// Problems: 3x3, stride 1, pad 1, output grid = input grid, Cg % GKS == 0, ncol % TN == 0, bf16
// (TN = 64: ncol of 64 columns, never split along K).
template <int MODE, int TN>
__global__ __launch_bounds__(256, 2) void gemm_conv_kernel(const ConvLaunch L) {
  using T = uint16_t;
  using G = GemmTile<TN>;
  constexpr int VE = 8;
  constexpr int GOPS = G::OPS;
  __shared__ __attribute__((aligned(16))) float smem[G::SMEM / 4];
  __shared__ __attribute__((aligned(16))) float2 pro_s[CONV_PRO_MAXC];
  __shared__ __attribute__((aligned(16))) float bn_s[MODE == MODE_BWD ? 7 * TN : 1];
  uint16_t* ops = (uint16_t*)smem;

  const int gi = find_group(L);
  const ConvProb& P = L.p[gi];
  const int local = blockIdx.x - P.tile_begin;
  const int ntile = P.tiles_m * P.tiles_n;
  const int ks = TN == 128 && P.ksplit > 1 ? P.ksplit : 1;   // workgroups per tile along K
  const int split = local / ntile;
  const int tl = local - split * ntile;
  const int tm = tl / P.tiles_n;
  const int tn = tl - tm * P.tiles_n;
  const int n0 = tn * TN;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int r32 = lane & 31, kh = lane >> 5;
  const int wr = TN == 128 ? wave >> 1 : wave, wc = TN == 128 ? wave & 1 : 0;
  const bool prologue = MODE == MODE_FWD && P.pro != nullptr;
  const bool bnmask = MODE == MODE_BWD && (P.flags & (EPI_BN_MASK | EPI_BN_APPLY));

  // loader geometry: thread tid moves 16-byte chunk ch of rows (and filter rows) lr + GLR h.  Per
  // row: the element offset of its own pixel (the tap offset is uniform: ((r - 1) W + s - 1) Cg in
  // the forward, mirrored in the data gradient) and a mask of the taps whose pixel is inside the image.
  const int ch = tid % GCH, lr = tid / GCH;
  const int PQ = P.P * P.Q;
  long abase[GLP];
  unsigned amask[GLP];
#pragma unroll
  for (int h = 0; h < GLP; ++h) {
    const int m = tm * GM + lr + GLR * h;
    const bool v = m < P.M;
    const int mm = v ? m : 0;
    const int n = div_l2(mm, PQ, P.pq_log2);
    const int rem = mm - n * PQ;
    const int p = div_l2(rem, P.Q, P.q_log2);
    const int q = rem - p * P.Q;
    abase[h] = (((long)n * P.H + p) * P.W + q) * P.Cg + 8 * ch;
    unsigned mk = 0;
#pragma unroll
    for (int t = 0; t < 9; ++t) {
      const int dr = MODE == MODE_FWD ? t / 3 - 1 : 1 - t / 3;
      const int dq = MODE == MODE_FWD ? t % 3 - 1 : 1 - t % 3;
      mk |= (v && (unsigned)(p + dr) < (unsigned)P.H && (unsigned)(q + dq) < (unsigned)P.W) ? 1u << t : 0u;
    }
    amask[h] = mk;
  }
  const T* wrow = (const T*)P.wmat + (long)(n0 + lr) * P.K + 8 * ch;   // ncol % TN == 0: all valid

  if (prologue)
    for (int c = tid; c < P.Cg; c += 256) pro_s[c] = make_float2(P.pro[c], P.pro[P.Cg + c]);
  if (bnmask && tid < TN) {
    const int col = n0 + tid;
#pragma unroll
    for (int k = 0; k < 4; ++k) bn_s[k * TN + tid] = P.bnst[k * P.ncol + col];
    if (P.flags & EPI_BN_APPLY) {
#pragma unroll
      for (int k = 0; k < 3; ++k) bn_s[(4 + k) * TN + tid] = P.coef[k * P.ncol + col];
    }
  }

  // K step s covers tap s / (Cg / GKS), channels (s % (Cg / GKS)) GKS .. + GKS - 1.  Loads are
  // issued for every step unconditionally (padding and rows past M from a clamped, valid address,
  // zeroed when stored), so that no branch separates a load from the MFMAs it overlaps.
  const T* const in = (const T*)P.in;
  const int W = P.W, Cg = P.Cg, Kt = P.K;
  // this workgroup's K steps: [s_begin, s_begin + nsteps) of the problem's Kt / GKS
  const int ktot = Kt / GKS;
  const int s_begin = split * ktot / ks;
  const int nsteps = (split + 1) * ktot / ks - s_begin;
  struct Set {
    uint4 a[GLP], b[G::LPB];
    unsigned ok;                                   // bit h: row h of A is inside the image
    int c;                                         // channel of the thread's chunk
  };
  auto gload = [&](int s, Set& R) {
    s = s_begin + (s < nsteps ? s : nsteps - 1);   // past the end: a repeat of the last step
    // channel chunk outer, tap inner: consecutive steps read the same channels of rows shifted by
    // one pixel or one image row, which the vector L1 of the CU serves again
    const int cb = s / 9, tap = s - 9 * cb;
    const int cs = cb * GKS;
    const int k0 = tap * Cg + cs;
    R.c = cs + 8 * ch;
    const int dr = MODE == MODE_FWD ? tap / 3 - 1 : 1 - tap / 3;
    const int dq = MODE == MODE_FWD ? tap % 3 - 1 : 1 - tap % 3;
    const long toff = ((long)dr * W + dq) * Cg + cs;
    R.ok = 0;
#pragma unroll
    for (int h = 0; h < GLP; ++h) {
      const bool ok = (amask[h] >> tap) & 1u;
      R.ok |= ok ? 1u << h : 0u;
      R.a[h] = *(const uint4*)(in + (ok ? abase[h] + toff : 0));
    }
#pragma unroll
    for (int h = 0; h < G::LPB; ++h) R.b[h] = *(const uint4*)(wrow + (long)GLR * h * Kt + k0);
  };
  // a step's chunks into LDS stage st (prologue: ReLU(x scale + shift) of the stored values;
  // padding and rows past M are zeros of the activated operand)
  auto lstore = [&](int st, const Set& R) {
    uint16_t* A = ops + st * GOPS;
    uint16_t* Bt = A + GM * GAS;
    float2 ps[VE];                                 // the chunk's (scale, shift): one channel set per step
    if (prologue) {
#pragma unroll
      for (int e = 0; e < VE; e += 2) {
        const float4 u = *(const float4*)&pro_s[R.c + e];
        ps[e] = make_float2(u.x, u.y);
        ps[e + 1] = make_float2(u.z, u.w);
      }
    }
#pragma unroll
    for (int h = 0; h < GLP; ++h) {
      const unsigned keep = 0u - ((R.ok >> h) & 1u);   // all ones for a row inside the image
      uint4 w = make_uint4(R.a[h].x & keep, R.a[h].y & keep, R.a[h].z & keep, R.a[h].w & keep);
      if (prologue) {
        Chunk<T> v;
        unpack_chunk<T>(w, v);
        float f[VE];
#pragma unroll
        for (int e = 0; e < VE; ++e) f[e] = fmaxf(fmaf(v.v[e], ps[e].x, ps[e].y), 0.0f);
        store_chunk<T>(&w, 0, f);
        w = make_uint4(w.x & keep, w.y & keep, w.z & keep, w.w & keep);
      }
      *(uint4*)(A + (lr + GLR * h) * GAS + 8 * ch) = w;
    }
#pragma unroll
    for (int h = 0; h < G::LPB; ++h) *(uint4*)(Bt + (lr + GLR * h) * GAS + 8 * ch) = R.b[h];
  };

  constexpr int MI = G::MI;
  f32x16 acc[MI][2];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  auto compute = [&](int st) {
    const uint16_t* A = ops + st * GOPS;
    const uint16_t* Bt = A + GM * GAS;
#pragma unroll
    for (int kk = 0; kk < GKS / 16; ++kk) {
      bf16x8 a[MI], b[2];
#pragma unroll
      for (int i = 0; i < MI; ++i)
        a[i] = *(const bf16x8*)(A + (wr * G::WROWS + 32 * i + r32) * GAS + 16 * kk + 8 * kh);
#pragma unroll
      for (int j = 0; j < 2; ++j)
        b[j] = *(const bf16x8*)(Bt + (wc * 64 + 32 * j + r32) * GAS + 16 * kk + 8 * kh);
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
    }
  };

  // Step s computes from stage s & 1.  Two register sets: while step s computes, step s + 1's
  // loads (issued a step earlier) are written to the other stage after the MFMAs and step s + 2's
  // are in flight.  Each half of the loop body is straight-line code.
  Set R0, R1;
  gload(0, R0);
  gload(1, R1);
  __syncthreads();                                 // prologue constants in LDS
  lstore(0, R0);
  __syncthreads();
  auto half = [&](int s, int st, Set& far, const Set& next) {
    gload(s + 2, far);
    __builtin_amdgcn_sched_barrier(0);
    compute(st);
    __builtin_amdgcn_sched_barrier(0);
    lstore(st ^ 1, next);
    __syncthreads();
  };
  int s = 0;
  for (; s + 1 < nsteps; s += 2) {
    half(s, 0, R0, R1);
    half(s + 1, 1, R1, R0);
  }
  if (s < nsteps) compute(0);                      // an odd step count: the last step
  __syncthreads();

  if (TN == 128 && ks > 1) {
    // a split of K: the raw fp32 tile to the partial buffer in the accumulators' own order, one
    // 32 x 32 block after the other (blocks by wave row, wave column, i, j); within a block the
    // float4 of lane l and row group g (rows 8 g + 4 (l / 32) .. + 3 of column l % 32) at g * 64 + l,
    // so each store writes 1 KB contiguously.  The epilogue runs once every split is done.
    float4* dst = (float4*)(P.kpart + ((long)split * ntile + tl) * (GM * GN));
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const int blk = ((wr * 2 + wc) * 2 + i) * 2 + j;
#pragma unroll
        for (int g = 0; g < 4; ++g)
          dst[blk * 256 + g * 64 + lane] =
              make_float4(acc[i % MI][j][4 * g], acc[i % MI][j][4 * g + 1], acc[i % MI][j][4 * g + 2],
                          acc[i % MI][j][4 * g + 3]);
      }
    return;
  }

  // stage the fp32 tile: D lane layout of the 32 x 32 MFMA (column r32, rows 8 (e / 4) + 4 kh + e % 4)
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e)
        smem[(wr * G::WROWS + 32 * i + 8 * (e >> 2) + 4 * kh + (e & 3)) * G::LDA + wc * 64 + 32 * j + r32] =
            acc[i][j][e];

  // streamed epilogue operands of the thread's chunks (as the other conv kernels)
  constexpr int ncc = TN / VE, rpp = 256 / ncc, NCH = GM / rpp;
  const int cc0 = (tid % ncc) * VE;
  const void* pf = (MODE == MODE_FWD) ? P.res
                   : ((P.flags & EPI_STORE_F32) ? nullptr : (bnmask ? P.zsrc : P.res));
  const void* pf2 = (MODE == MODE_FWD) ? P.ext : ((P.flags & EPI_BN_APPLY) ? P.res : nullptr);
  uint4 pre[NCH], pre2[NCH];
#pragma unroll
  for (int k = 0; k < NCH; ++k) {
    const int m = tm * GM + tid / ncc + k * rpp;
    const long o = (long)m * P.ncol + n0 + cc0;
    pre[k] = (pf != nullptr && m < P.M) ? *(const uint4*)((const T*)pf + o) : make_uint4(0, 0, 0, 0);
    pre2[k] = (pf2 != nullptr && m < P.M) ? *(const uint4*)((const T*)pf2 + o) : make_uint4(0, 0, 0, 0);
  }
  __syncthreads();
  conv_epilogue<T, MODE, GM, TN, G::LDA, TN>(P, smem, (float*)pro_s, bn_s, tm, n0, pre, pre2);
}

// Second pass of the split problems: one workgroup per slab of GEMM_RBN = 16 columns of a 128 x 128
// tile (half of one 32-column block column of the first pass's order).  Thread t sums, in split
// order, the float4s f = t and t + 256 of the slab (f: lane within the half, its row-group half, row
// group, i, wave row), eight splits' loads in flight per round (repeats of the last split past
// the end); the sums go to the staged row-major slab, then the slab's epilogue.
template <int MODE>
__global__ __launch_bounds__(256) void gemm_reduce_kernel(const ConvLaunch L) {
  using T = uint16_t;
  constexpr int VE = 8, RB = GEMM_RBN, LDA = RB + 4, CPT = GN / RB;
  constexpr int ACCW = 2 * 256 * VE + 512;       // the epilogue's stats scratch exceeds the staged slab
  static_assert(GM * 2 == 256 && RB == 16 && CPT == 8, "slab layout");
  __shared__ __attribute__((aligned(16))) float smem[ACCW > GM * LDA ? ACCW : GM * LDA];
  __shared__ __attribute__((aligned(16))) float piv_s[RB];
  __shared__ __attribute__((aligned(16))) float bn_s[MODE == MODE_BWD ? 7 * RB : 1];

  const int gi = find_group(L);
  const ConvProb& P = L.p[gi];
  const int local = blockIdx.x - P.tile_begin;
  const int tl = local / CPT;
  const int cs = local - tl * CPT;
  const int ntile = P.tiles_m * P.tiles_n;
  const int tm = tl / P.tiles_n;
  const int cn = (tl - tm * P.tiles_n) * GN + cs * RB;   // the slab's first column
  const int tid = threadIdx.x;
  const bool bnmask = MODE == MODE_BWD && (P.flags & (EPI_BN_MASK | EPI_BN_APPLY));
  // every global load is issued before the first LDS write: the BN constants of the slab's
  // columns, the epilogue operands, then the partials
  const bool bnload = bnmask && tid < RB;
  float bnv[7];
  if (bnload) {
#pragma unroll
    for (int k = 0; k < 4; ++k) bnv[k] = P.bnst[k * P.ncol + cn + tid];
#pragma unroll
    for (int k = 0; k < 3; ++k) bnv[4 + k] = (P.flags & EPI_BN_APPLY) ? P.coef[k * P.ncol + cn + tid] : 0.f;
  }
  const void* pf = (MODE == MODE_FWD) ? P.res
                   : ((P.flags & EPI_STORE_F32) ? nullptr : (bnmask ? P.zsrc : P.res));
  const void* pf2 = (MODE == MODE_FWD) ? P.ext : ((P.flags & EPI_BN_APPLY) ? P.res : nullptr);
  uint4 pre[1], pre2[1];
  {
    const int m = tm * GM + (tid >> 1);            // the epilogue's chunk: row tid / 2, 8 columns
    const long o = (long)m * P.ncol + cn + (tid & 1) * VE;
    pre[0] = (pf != nullptr && m < P.M) ? *(const uint4*)((const T*)pf + o) : make_uint4(0, 0, 0, 0);
    pre2[0] = (pf2 != nullptr && m < P.M) ? *(const uint4*)((const T*)pf2 + o) : make_uint4(0, 0, 0, 0);
  }
  // the slab in the first pass's order: wave column wc, block column j, half h of the 32 columns
  const int wc = cs >> 2, j = (cs >> 1) & 1, h = cs & 1;
  int off[2], row[2];
  const int l16 = tid & 15;
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int f = tid + 256 * u;
    const int kh = (f >> 4) & 1, g = (f >> 5) & 3, i = (f >> 7) & 1, wr = f >> 8;
    off[u] = (((wr * 2 + wc) * 2 + i) * 2 + j) * 256 + g * 64 + kh * 32 + h * 16 + l16;
    row[u] = wr * 64 + 32 * i + 8 * g + 4 * kh;
  }
  const float4* src = (const float4*)(P.kpart + (long)tl * (GM * GN));
  const long ss = (long)ntile * (GM * GN / 4);
  const int S = P.ksplit;
  float4 a[2] = {make_float4(0.f, 0.f, 0.f, 0.f), make_float4(0.f, 0.f, 0.f, 0.f)};
  for (int k0 = 0; k0 < S; k0 += 8) {
    float4 v[8][2];
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      const long k = min(k0 + w, S - 1);
      v[w][0] = src[k * ss + off[0]];
      v[w][1] = src[k * ss + off[1]];
    }
#pragma unroll
    for (int w = 0; w < 8; ++w) {
      if (k0 + w < S) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          a[u].x += v[w][u].x; a[u].y += v[w][u].y; a[u].z += v[w][u].z; a[u].w += v[w][u].w;
        }
      }
    }
  }
  if (bnload) {
#pragma unroll
    for (int k = 0; k < 7; ++k) bn_s[k * RB + tid] = bnv[k];
  }
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    smem[(row[u] + 0) * LDA + l16] = a[u].x;
    smem[(row[u] + 1) * LDA + l16] = a[u].y;
    smem[(row[u] + 2) * LDA + l16] = a[u].z;
    smem[(row[u] + 3) * LDA + l16] = a[u].w;
  }
  __syncthreads();
  conv_epilogue<T, MODE, GM, RB, LDA, RB>(P, smem, piv_s, bn_s, tm, cn, pre, pre2);
}

int launch_gemm_reduce(const ConvLaunch& L, int tiles, int mode, hipStream_t s) {   // tiles: slabs
  if (mode == MODE_FWD)
    hipLaunchKernelGGL(gemm_reduce_kernel<MODE_FWD>, dim3(tiles), dim3(256), 0, s, L);
  else
    hipLaunchKernelGGL(gemm_reduce_kernel<MODE_BWD>, dim3(tiles), dim3(256), 0, s, L);
  return (int)hipGetLastError();
}

int launch_gemm(const ConvLaunch& L, int tiles, int mode, int tn, hipStream_t s) {
  if (tn == 64) {
    if (mode == MODE_FWD)
      hipLaunchKernelGGL((gemm_conv_kernel<MODE_FWD, 64>), dim3(tiles), dim3(256), 0, s, L);
    else
      hipLaunchKernelGGL((gemm_conv_kernel<MODE_BWD, 64>), dim3(tiles), dim3(256), 0, s, L);
  } else {
    if (mode == MODE_FWD)
      hipLaunchKernelGGL((gemm_conv_kernel<MODE_FWD, 128>), dim3(tiles), dim3(256), 0, s, L);
    else
      hipLaunchKernelGGL((gemm_conv_kernel<MODE_BWD, 128>), dim3(tiles), dim3(256), 0, s, L);
  }
  return (int)hipGetLastError();
}

// ------------------------------------------------------------------------------------------------
// Weight gradient of a wide 3x3 / stride 1 / pad 1 bf16 convolution as a GEMM over the output
// pixels: dW[co][(tap, c)] = sum_m g[m][co] * act(in)[pixel(m) + tap][c] (the weight gradient of the
// layers of Table vgg), TC output channels x TK filter columns (one tap's TK input channels) per
// workgroup, TC and TK 128 or 64, split over m.  Stages of 64 pixels: the output-gradient rows and
// the gathered input rows (BN prologue applied on the way, zeros outside the image) are staged
// m-major in LDS (rows padded by 16 elements: the four rows of a transposed read fall on distinct
// banks; in 128-column operands rows 8 .. 15 of every 16 are rotated by 64 columns, so that the two
// lane groups of a half-wave, 8 rows apart, read disjoint banks), read as MFMA fragments with the gfx950 transposed LDS read; four waves of
// (TC / 2) x (TK / 2) (16x16x32 MFMAs).  Loads run two stages ahead in two register sets; two LDS
// stages.  The fp32 partial tile goes to part[split][co][K] for the split-K column reduce.
// ------------------------------------------------------------------------------------------------
namespace {
constexpr int WGM_KC = 64;                  // pixels per stage

typedef short wv4s16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) wv4s16 lds_wv4s16;

// LDS column of element column c of row r of a W-column operand (W = 128: rows with bit 3 set
// rotated by 64 columns; measured: 128 x 128 tiles 2010 -> 1956 us per VGG-224 launch, while the
// 64-column operands, given 144-element rows for the same rotation, ran 1732 -> 2721 us)
template <int W>
__device__ __forceinline__ int wgm_col(int r, int c) { return W == 128 ? (c + ((r & 8) << 3)) & 127 : c; }

// the 16x16x32 MFMA fragment of 16 columns (cbase ..) over 8 rows (row0 .. row0 + 7, row0 a multiple
// of 8) of an m-major W-column tile of row stride RS: lane group rows 4 (r16 / 4) apart by the
// transposed read
template <int W, int RS>
__device__ __forceinline__ void tr_frag(const uint16_t* base, int row0, int cbase, int r16, Frag<uint16_t>& f) {
  const uint16_t* p0 = base + (row0 + (r16 >> 2)) * RS + wgm_col<W>(row0, cbase + 4 * (r16 & 3));
  const wv4s16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_wv4s16*)p0);
  const wv4s16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_wv4s16*)(p0 + 4 * RS));
  const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
  f.from_raw(make_uint4(l2.x, l2.y, h2.x, h2.y));
}

// loader geometry of a W-column m-major operand: 16-byte chunks, 256 threads
template <int W>
struct WgmOp {
  static constexpr int CPR = W / 8;              // chunks per row
  static constexpr int RPP = 256 / CPR;          // rows per pass
  static constexpr int NP = WGM_KC / RPP;        // passes per stage
  static constexpr int RS = W + 16;              // LDS row stride (elements)
  static_assert((W == 64 || W == 128) && RS * 2 % 16 == 0, "16-byte aligned rows");
};
}  // namespace

template <int TC, int TK>
__global__ __launch_bounds__(256, 2) void wgrad_gemm_kernel(const WgradLaunch L) {
  using T = uint16_t;
  using OG = WgmOp<TC>;
  using OA = WgmOp<TK>;
  constexpr int VE = 8;
  constexpr int STG = WGM_KC * (OG::RS + OA::RS);   // elements per LDS stage (gradient, then input)
  constexpr int NI = TC / 32, NJ = TK / 32;         // 16-row MFMA blocks per wave
  static_assert(OG::NP <= 4 && OA::NP <= 4 && OG::NP * OG::RPP == WGM_KC && OA::NP * OA::RPP == WGM_KC,
                "loader");
  __shared__ __attribute__((aligned(16))) uint16_t smem[2 * STG];
  __shared__ float2 pro_s[TK];
  const int gi = find_group(L);
  const WgradProb& P = L.p[gi];
  const int local = blockIdx.x - P.tile_begin;
  // Workgroups go to the eight XCDs round-robin by blockIdx, and each XCD has its own L2.  The
  // tiles of one split (every tap and output-channel tile over the same pixels) read the same
  // gradient rows and the same input rows shifted by a pixel.  For 64-channel output tiles (L2 hit
  // rate 6 % in plain order) the first 8 floor(splits / 8) splits are grouped by XCD: local index
  // 8 q + x takes split x + 8 (q / W), tile q % W (W tiles per split), so all of a split's tiles
  // share one XCD (19 % faster there; the 128-channel tiles, 60 % hits already, ran 3 % slower so).
  // The remaining splits, and every split of 128-channel tiles, in plain order.
  const int W = P.tiles_co * P.tiles_k;
  const int S8 = TC == 64 ? P.splits & ~7 : 0;
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
  const int tk = t % P.tiles_k;
  const int tco = t / P.tiles_k;
  const int co0 = tco * TC, k0 = tk * TK;
  const int tap = k0 / P.Cg, c0 = k0 - tap * P.Cg;      // (Cg a multiple of TK)
  const int dr = tap / 3 - 1, dc = tap - 3 * (tap / 3) - 1;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int r16 = lane & 15, grp = lane >> 4;
  const int wr = wave >> 1, wc = wave & 1;
  const int m_begin = split * P.mchunk;
  const int m_end = min(P.M, m_begin + P.mchunk);
  const int nst = (m_end - m_begin + WGM_KC - 1) / WGM_KC;
  const bool prologue = P.pro != nullptr;
  if (tid < TK) pro_s[tid] = prologue ? make_float2(P.pro[c0 + tid], P.pro[P.Cg + c0 + tid]) : make_float2(1.f, 0.f);

  // loaders: gradient chunk h of a stage is row lrg + RPP h, 16-byte column lcg; input chunk h row
  // lra + RPP h, column lca.  Stride 1 and equal maps: the input pixel of output pixel m at the tap is
  // m + dr W + dc; the input row's (p, q) in its image, needed only for the in-image test, advance by
  // WGM_KC pixels a stage as a mixed-radix count
  const int lcg = (tid % OG::CPR) * VE, lrg = tid / OG::CPR;
  const int lca = (tid % OA::CPR) * VE, lra = tid / OA::CPR;
  const int PQ = P.P * P.Q;
  const T* gbase = (const T*)P.g + co0 + lcg;
  const T* ibase = (const T*)P.in + c0 + lca;
  const int toff = dr * P.W + dc;
  const int sq = WGM_KC % P.Q, sp = (WGM_KC / P.Q) % P.P;    // a stage's step in (p, q)
  int rp[OA::NP], rqq[OA::NP];
#pragma unroll
  for (int h = 0; h < OA::NP; ++h) {
    const int pix = (m_begin + lra + OA::RPP * h) % PQ;     // (once per workgroup)
    rp[h] = pix / P.Q;
    rqq[h] = pix - rp[h] * P.Q;
  }
  int lstage = 0;                                            // the stage (rp, rqq) describe
  struct Set {
    uint4 g[OG::NP], a[OA::NP];
    unsigned ok;       // bit h: gradient row h exists; bit 4 + h: input row h's pixel exists
  };
  auto load = [&](int s, Set& R) {
    const int sc = s < nst ? s : nst - 1;                    // past the end: a repeat, masked
    if (sc != lstage) {                                      // (stages are loaded in order)
#pragma unroll
      for (int h = 0; h < OA::NP; ++h) {
        int q = rqq[h] + sq, p = rp[h] + sp;
        if (q >= P.Q) { q -= P.Q; ++p; }
        if (p >= P.P) p -= P.P;
        rqq[h] = q;
        rp[h] = p;
      }
      lstage = sc;
    }
    const int mc = m_begin + sc * WGM_KC;
    R.ok = 0;
#pragma unroll
    for (int h = 0; h < OG::NP; ++h) {
      const int m = mc + lrg + OG::RPP * h;
      const bool vm = s < nst && m < m_end;
      R.g[h] = *(const uint4*)(gbase + (vm ? (long)m * P.Co : 0));
      R.ok |= (vm ? 1u : 0u) << h;
    }
#pragma unroll
    for (int h = 0; h < OA::NP; ++h) {
      const int m = mc + lra + OA::RPP * h;
      const bool vm = s < nst && m < m_end;
      const int ih = rp[h] + dr, iw = rqq[h] + dc;
      const bool vi = vm && (unsigned)ih < (unsigned)P.H && (unsigned)iw < (unsigned)P.W;
      R.a[h] = *(const uint4*)(ibase + (vi ? (long)(m + toff) * P.Cg : 0));
      R.ok |= (vi ? 1u : 0u) << (4 + h);
    }
  };
  auto store = [&](int st, const Set& R) {
    uint16_t* G = smem + st * STG;
    uint16_t* A = G + WGM_KC * OG::RS;
#pragma unroll
    for (int h = 0; h < OG::NP; ++h) {
      const unsigned kg = 0u - ((R.ok >> h) & 1u);
      const int r = lrg + OG::RPP * h;                      // (rows 16-byte aligned: 16-byte writes)
      const int o = r * OG::RS + wgm_col<TC>(r, lcg);
      *(uint4*)(G + o) = make_uint4(R.g[h].x & kg, R.g[h].y & kg, R.g[h].z & kg, R.g[h].w & kg);
    }
#pragma unroll
    for (int h = 0; h < OA::NP; ++h) {
      const unsigned ka = 0u - ((R.ok >> (4 + h)) & 1u);
      uint4 w = R.a[h];
      if (prologue) {
        Chunk<T> v;
        unpack_chunk<T>(w, v);
        float f[VE];
#pragma unroll
        for (int e = 0; e < VE; ++e) f[e] = fmaxf(fmaf(v.v[e], pro_s[lca + e].x, pro_s[lca + e].y), 0.0f);
        store_chunk<T>(&w, 0, f);
      }
      const int r = lra + OA::RPP * h;
      const int o = r * OA::RS + wgm_col<TK>(r, lca);
      *(uint4*)(A + o) = make_uint4(w.x & ka, w.y & ka, w.z & ka, w.w & ka);
    }
  };
  f32x4 acc[NI][NJ];
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  // The next sub-step's fragments are read into the registers of the current one as soon as their
  // last MFMA has issued (A fragment i after row i, B fragment j after the last row's MFMA j), so
  // that the reads overlap the remaining MFMAs.
  auto compute = [&](int st) {
    const uint16_t* G = smem + st * STG;
    const uint16_t* A = G + WGM_KC * OG::RS;
    Frag<T> a[NI], b[NJ];
#pragma unroll
    for (int i = 0; i < NI; ++i) tr_frag<TC, OG::RS>(G, VE * grp, wr * (TC / 2) + 16 * i, r16, a[i]);
#pragma unroll
    for (int j = 0; j < NJ; ++j) tr_frag<TK, OA::RS>(A, VE * grp, wc * (TK / 2) + 16 * j, r16, b[j]);
#pragma unroll
    for (int sub = 0; sub < WGM_KC / 32; ++sub) {
      const bool more = sub + 1 < WGM_KC / 32;
      const int row1 = (sub + 1) * 32 + VE * grp;
#pragma unroll
      for (int i = 0; i < NI; ++i) {
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
          mma(a[i], b[j], acc[i][j]);
          if (more && i == NI - 1) tr_frag<TK, OA::RS>(A, row1, wc * (TK / 2) + 16 * j, r16, b[j]);
        }
        if (more) tr_frag<TC, OG::RS>(G, row1, wr * (TC / 2) + 16 * i, r16, a[i]);
      }
    }
  };

  Set R0, R1;
  load(0, R0);
  load(1, R1);
  __syncthreads();                                   // pro_s
  store(0, R0);
  __syncthreads();
  auto half = [&](int s, int st, Set& far, const Set& next) {
    load(s + 2, far);
    __builtin_amdgcn_sched_barrier(0);
    compute(st);
    __builtin_amdgcn_sched_barrier(0);
    store(st ^ 1, next);
    __syncthreads();
  };
  int s = 0;
  for (; s + 1 < nst; s += 2) {
    half(s, 0, R0, R1);
    half(s + 1, 1, R1, R0);
  }
  if (s < nst) compute(0);

  // the partial tile: lane (r16, grp) holds rows 4 grp + e of each 16 x 16 block
#pragma unroll
  for (int i = 0; i < NI; ++i)
#pragma unroll
    for (int j = 0; j < NJ; ++j)
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int co = co0 + wr * (TC / 2) + 16 * i + 4 * grp + e;
        const int k = k0 + wc * (TK / 2) + 16 * j + r16;
        P.part[((long)split * P.Co + co) * P.K + k] = acc[i][j][e];
      }
}

int launch_wgrad_gemm(const WgradLaunch& L, int tiles, int tc, int tk, hipStream_t s) {
  if (tc == 128 && tk == 128)
    hipLaunchKernelGGL((wgrad_gemm_kernel<128, 128>), dim3(tiles), dim3(256), 0, s, L);
  else if (tc == 128 && tk == 64)
    hipLaunchKernelGGL((wgrad_gemm_kernel<128, 64>), dim3(tiles), dim3(256), 0, s, L);
  else if (tc == 64 && tk == 128)
    hipLaunchKernelGGL((wgrad_gemm_kernel<64, 128>), dim3(tiles), dim3(256), 0, s, L);
  else if (tc == 64 && tk == 64)
    hipLaunchKernelGGL((wgrad_gemm_kernel<64, 64>), dim3(tiles), dim3(256), 0, s, L);
  else
    return (int)hipErrorInvalidValue;
  return (int)hipGetLastError();
}

}  // namespace pnn
