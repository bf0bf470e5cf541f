// Internal declarations of libpnn: grouped-launch problem descriptors shared by the host plan
// code and the gfx950 kernels, plus the launchers.
//
// A grouped launch carries up to PNN_MAXG (for small problem records more, within the 4 KB of
// kernel arguments) independent problems by value in its kernel arguments (the N fine
// sub-networks of one depth level are the groups of one launch).  Every problem owns a contiguous
// range [tile_begin, tile_begin + tiles) of the launch's workgroups.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

struct pnn_plan;

#define PNN_MAXG 20
#define PNN_BN_EPS 1e-5f

namespace pnn {

enum { MODE_FWD = 0, MODE_BWD = 1 };

// conv epilogue flags
enum {
  EPI_STATS = 1,      // FWD: per-column sum / sum of squares of the stored output -> part
  EPI_BN_MASK = 2,    // BWD: dbn = v * [ReLU(BN(z)) > 0] stored, sums of dbn and dbn * xhat -> part
  EPI_STORE_F32 = 4,  // BWD: v stored as float to out32 (first of two consumers of one BN)
  EPI_ACC_IN = 8,     // BWD: v += acc_in before the epilogue
  EPI_NO_STORE = 16,  // BWD + EPI_BN_MASK: BN sums only, dbn is not stored
  EPI_BN_APPLY = 32,  // BWD: dbn = rnd(v * mask) as for EPI_BN_MASK, then the BN backward apply
                      // out = A dbn + B z + K [+ res] (coefficients coef [3][ncol]); no sums
  EPI_PW_WGRAD = 64,  // pw_kernel BWD / bnsum_kernel: also the convolution's weight gradient from
                      // the same tiles, split-K partial row tm of out32 [tiles_m][K][ncol]
                      // (g^T . ReLU(BN(z)))
  EPI_BN_FUSE = 128,  // FWD + EPI_STATS: the producer also finalises the BN statistics from the
                      // partial rows (bn_fwd_fuse: the last workgroup of a row group folds the
                      // group, the last group the whole column) into bn_stats; no column-reduce pass
};

// Implicit-GEMM convolution problem.  FWD: out[m][n] = sum_k A[m][k] wmat[n][k] with
// A[m][(r,s,c)] = act(in)[pixel(m) + tap(r,s)][c].  BWD (data gradient): the same with the
// transposed-convolution gather: A = output gradient, wmat = filter transposed to [c_in][r][s][c_out].
struct ConvProb {
  const void* in;       // gathered tensor [B][H][W][Cg] (storage type)
  const void* wmat;     // [ncol][K], K contiguous (storage type)
  void* out;            // [M][ncol] storage type
  const void* res;      // addend [M][ncol] (nullable); BWD: the skip gradient
  const void* ext;      // second addend [M][ncol] (nullable)
  const float* pro;     // FWD prologue scale[Cg], shift[Cg]: A = ReLU(x * scale + shift) (nullable)
  float* part;          // per-tile column partial sums [tiles_m][ncol][2]
  union {
    const void* zsrc;   // BWD + EPI_BN_MASK: BN input z [M][ncol]
    unsigned* bn_cnt;   // FWD + EPI_BN_FUSE: arrival counters (bn_fwd_fuse), zero at launch
  };
  union {
    const float* bnst;      // BWD + EPI_BN_MASK: mean, invstd, scale, shift [4][ncol]
    const float* bn_gamma;  // FWD + EPI_BN_FUSE: gamma [ncol], then beta [ncol]
  };
  const float* acc_in;  // EPI_ACC_IN: [M][ncol] float
  const float* coef;    // EPI_BN_APPLY: A, B, K [3][ncol]
  union {
    float* out32;       // EPI_STORE_F32: [M][ncol] float
    float* bn_stats;    // FWD + EPI_BN_FUSE: mean, invstd, scale, shift [4][ncol] (written)
  };
  float* kpart;         // GEMM kernel, ksplit > 1: fp32 partial tiles [ksplit][tiles][GEMM_BM][GEMM_BN]
  int B, H, W, Cg;      // gathered tensor
  int P, Q;             // output pixel grid (M = B * P * Q)
  int ncol;
  int k, stride, pad;   // forward convolution geometry (BWD gathers through its transpose)
  int M, K;
  int tiles_m, tiles_n, wn, wm;   // tiles; column and row sub-tiles per wave
  int flags;
  int ksplit;           // GEMM kernel: K split over this many workgroups per tile (<= 1: none)
  int cg_log2;          // log2(Cg) when Cg is a power of two, else -1
  int q_log2, pq_log2;  // log2(Q), log2(P*Q) when powers of two, else -1
  int tile_begin;
};
// Launch records that open with a lookup table tb (tb[0]: problem count; tb[p], p >= 1: first
// workgroup of problem p, non-decreasing, problems without tiles sharing the next one's begin)
template <typename L, typename = void> struct HasTb : std::false_type {};
template <typename L> struct HasTb<L, std::void_t<decltype(std::declval<L>().tb)>> : std::true_type {};

struct ConvLaunch {
  int tb[PNN_MAXG];   // [0]: problem count; [p >= 1]: first workgroup of problem p (the lookup table)
  int n;
  ConvProb p[PNN_MAXG];
};

// Weight gradient: part[split][co][kk] = sum over the split's rows m of g[m][co] * A[m][kk].
struct WgradProb {
  const void* g;        // [M][Co]
  const void* in;       // [B][H][W][Cg]
  const float* pro;     // prologue scale / shift (nullable)
  float* part;          // [splits][Co][K] float
  int B, H, W, Cg, P, Q, Co, k, stride, pad, M, K;
  int wr;               // tile = (16 wr) output channels x 64 filter columns
  int gtc, gtk;         // GEMM kernel tile: output channels, filter columns (128 or 64 each)
  int tiles_co, tiles_k, splits, mchunk;
  int cg_log2, q_log2, pq_log2;   // as in ConvProb
  int tile_begin;
};
struct WgradLaunch {
  int tb[PNN_MAXG];   // [0]: problem count; [p >= 1]: first workgroup of problem p (the lookup table)
  int n;
  WgradProb p[PNN_MAXG];
};

// Column reduction of tile partials part[rows][ncols] in a fixed order (fp64 sums), fused with what
// the sums are for:
//   RED_SUM     dst[c] = sum_r part[r][c]                               (split-K weight gradients;
//               ncols even, two columns per thread, rows split over 2^rl_log2 lanes)
//   RED_BN_FWD  ncols = 2C, part[r][c][2] = (mean, sum of squared deviations from it) of the rowh
//               rows of partial row r (the last one ragged) -> mean, invstd, scale, shift [4][C]
//   RED_BN_BWD  ncols = 2C, part[r][c][2] = (sum dbn, sum dbn*xhat) -> dbeta, dgamma and the
//               apply coefficients c1 = gamma * invstd, mb = dbeta / M, mbx = dgamma / M  [3][C]
enum { RED_SUM = 0, RED_BN_FWD = 1, RED_BN_BWD = 2 };
struct ColRedProb {
  const float* part;
  float* dst;            // RED_SUM
  const float* gamma;    // BN modes
  const float* beta;     // RED_BN_FWD
  float* stats;          // RED_BN_FWD: written; RED_BN_BWD: read (invstd)
  float* dgamma;         // RED_BN_BWD
  float* dbeta;
  float* coef;
  long count;            // BN: number of rows M of the normalised tensor
  int rows, ncols, mode;
  int rl_log2;           // RED_SUM: log2 of the row lanes per column pair (0..5)
  int rowh;              // RED_BN_FWD: rows of the normalised tensor per partial row
  int tile_begin;
};
struct ColRedLaunch {
  int tb[40];   // [0]: problem count; [p >= 1]: first workgroup of problem p (the lookup table)
  int n;
  ColRedProb p[40];
};
constexpr int RED_COLS = 32;       // columns per column-reduce workgroup
constexpr int RED_LANES = 32;      // row lanes per column (1024 threads)
// RED_SUM row lanes: about eight rows per lane, at most 32 lanes
inline int red_sum_rl_log2(int rows) {
  int l = 0;
  while (l < 5 && (8 << l) < rows) ++l;
  return l;
}
inline int colred_tiles(int ncols, int mode, int rl_log2) {
  const int cols = mode == RED_SUM ? (2048 >> rl_log2) : RED_COLS;
  return (ncols + cols - 1) / cols;
}

// Column statistics of a stored tensor [M][C] (BN of a segment input).
struct ColStatProb {
  const void* x;
  float* part;          // [tiles][C][2]
  const float* gamma;   // fuse: gamma [C], then beta [C]
  float* stats;         // fuse: mean, invstd, scale, shift [4][C] (written)
  unsigned* cnt;        // fuse: arrival counters (bn_fwd_fuse), zero at launch
  long M;
  int C;
  int fuse;             // finalise the statistics as EPI_BN_FUSE does
  int tile_begin;
};
struct ColStatLaunch {
  int tb[PNN_MAXG];   // [0]: problem count; [p >= 1]: first workgroup of problem p (the lookup table)
  int n;
  ColStatProb p[PNN_MAXG];
};

// out = skip + c1 * (dbn - mb - xhat * mbx), xhat = (z - mean) * invstd  (BN backward apply).
struct BnApplyProb {
  const void* dbn;
  const void* z;
  const void* skip;     // nullable
  void* out;
  const float* stats;
  const float* coef;
  long n;
  int C;
  int tile_begin;
};
struct BnApplyLaunch {
  int tb[60];   // [0]: problem count; [p >= 1]: first workgroup of problem p (the lookup table)
  int n;
  BnApplyProb p[60];
};

// bnact: out = pool(ReLU(z * scale + shift)) [+ res] [+ ext]  (pool 0 or 2x2/2)
// bnact backward: dbn[z] = [y > 0] * (routed g), with per-tile sums of dbn and dbn * xhat.
struct BnActProb {
  const void* z;
  void* out;            // FWD: pooled output; BWD: dbn (z shaped)
  const void* res;      // FWD addend (nullable)
  const void* ext;      // FWD addend (nullable)
  const void* g;        // BWD: gradient of the output
  const float* stats;
  float* part;          // BWD: [tiles][C][2]
  int B, H, W, C, pool;
  long n_out;           // output pixels (B * Ho * Wo)
  int pix;              // output pixels per workgroup (BWD: BNACT_PIX, the partial rows' pixels)
  int tile_begin;
};
struct BnActLaunch {
  int tb[PNN_MAXG];   // [0]: problem count; [p >= 1]: first workgroup of problem p (the lookup table)
  int n;
  BnActProb p[PNN_MAXG];
};

// Elementwise / small kernels.
struct MaxPool3Prob {     // 256 * ve outputs per workgroup, ve per thread (1, or a 16-byte chunk)
  const void* x;
  void* y;
  int B, H, W, C, Ho, Wo;
  int ve;
  int tile_begin;
};
struct MaxPool3Launch {
  int tb[PNN_MAXG];   // [0]: problem count; [p >= 1]: first workgroup of problem p (the lookup table)
  int n;
  MaxPool3Prob p[PNN_MAXG];
};

struct TransposeProb {   // wt[c][r][s][o] = w[o][r][s][c]; T * ceil(O / 64) * ceil(C / 64) tiles
  const void* w;
  void* wt;
  int O, T, C;           // T = k * k taps
  int tile_begin;
};
struct TransposeLaunch {   // (no lookup table: 120 problems fill the argument space)
  int n;
  TransposeProb p[120];
};

struct AxpyProb {        // out = a - b (rounded to storage); partial sum of squares (nullable)
  const void* a;
  const void* b;
  void* out;
  float* sq_part;        // [tiles]
  long n;
  int tile_begin;
};
struct AxpyLaunch {
  int tb[PNN_MAXG];   // [0]: problem count; [p >= 1]: first workgroup of problem p (the lookup table)
  int n;
  unsigned* flag = nullptr;   // set to 1 when an output is not finite (nullable)
  AxpyProb p[PNN_MAXG];
};
// non-finite flags (uint32 words in scratch): [0] combine output r_j, [1] head loss / dW / db
constexpr int PNN_NFLAGS = 2;
int launch_flags_clear(unsigned* flags, hipStream_t s);

// SGD with momentum over a list of parameter tensors.  Entry e covers count elements at byte
// offset p_off of params[seg] and g_off of grads[seg] / momentum[seg]; workgroups
// [chunk0, chunk0 + ceil(count / SGD_CHUNK)) of the launch update it.
struct SgdEnt {
  uint32_t p_off, g_off, count, chunk0;
  uint16_t seg, f32;     // f32: parameters stored as float (else the plan's storage type)
};
constexpr int SGD_MAXT = 180;      // entries per launch
constexpr int SGD_MAXS = 8;        // segments per launch
constexpr int SGD_CHUNK = 2048;    // elements per workgroup
// m[seg] (nullable): fp32 master copy of the segment's storage-type filters, laid out like the
// gradient buffer; the update reads the master (or, with init, the stored filters) and writes both.
struct SgdLaunch {
  int nt, nesterov, init;
  float lr, mu, wd;
  void* p[SGD_MAXS];
  const float* g[SGD_MAXS];
  float* v[SGD_MAXS];
  float* m[SGD_MAXS];
  SgdEnt e[SGD_MAXT];
};
int launch_sgd(const SgdLaunch& L, int tiles, int dtype, hipStream_t s);

// Resident forward of a run of pre-activation bottleneck units (k_unit.hip): identity skip, stride
// 1, UNIT_H x UNIT_W maps, UNIT_C channels squeezed to UNIT_MID.  One workgroup per image of a
// sub-network ("job"); unit u's tensors sit at the first unit's byte offsets plus u times the
// launch's strides.
constexpr int UNIT_H = 32, UNIT_W = 32, UNIT_C = 64, UNIT_MID = 16;
constexpr int UNIT_WAVES = 8;       // waves per workgroup (one image)
constexpr int UNIT_MAXJ = 8;
// Barrier words at the start of the unit scratch (uint32): [0] error flag (a wait gave up), [1]
// barriers completed; job j's arrival counter and generation each on a 128-byte line of its own.
constexpr int UNIT_SYNC_BYTES = 4096;
__host__ __device__ constexpr int unit_sync_word(int job, int which) { return 64 * (job + 1) + 32 * which; }
static_assert(unit_sync_word(UNIT_MAXJ - 1, 1) * 4 + 4 <= UNIT_SYNC_BYTES, "unit barrier words");
struct UnitJob {
  const void* x_in;          // input of the first unit [B][H][W][C]
  const char* params;        // the segment's parameter buffer
  char* saved;               // the segment's saved workspace
  void* y_out;               // the segment output (the last unit's output when it has no BN)
  float* part;               // per-image statistics: z1 [B][MID][2], z2 [B][MID][2], x [B][C][2]
  int nu;                    // units
  int wg_begin;              // first workgroup of the job (one per image)
  unsigned w1, w2, w3;       // filters of the first unit's three convolutions (params)
  unsigned g1, g2, g3;       // gamma | beta of BN(x), BN(z1), BN(z2) (params)
  unsigned z1, z2, xo;       // z1, z2 and output slots of the first unit (saved)
  unsigned s1, s2, s3;       // BN statistics of BN(x), BN(z1), BN(z2) (saved)
  unsigned gN, sN;           // BN of the last unit's output (params, saved); 0xffffffff: none
};
struct UnitLaunch {
  int n, B, nu_max, nwg;
  unsigned dw, dg, dz, ds;   // per-unit strides: filters, BN parameters, slots, statistics
  unsigned* sync;            // barrier words (UNIT_SYNC_BYTES)
  UnitJob j[UNIT_MAXJ];
};
int launch_unit_reset(unsigned* sync, hipStream_t s);
int launch_unit_fwd(const UnitLaunch& L, hipStream_t s);
int unit_fwd_occupancy();    // workgroups of the resident kernel that fit the device at once

// gk: 0 = pointwise (1x1, stride 1, pad 0), 1 = vector gather, 2 = element-wise gather,
//     3 = 3x3 / stride 1 / pad 1 through an LDS halo tile;
// wn: 16-column sub-tiles per wave (1, 2, 4) shared by every problem of the launch
// every launch record fits the 4 KB of kernel arguments
static_assert(sizeof(ConvLaunch) <= 4096 && sizeof(WgradLaunch) <= 4096 && sizeof(ColRedLaunch) <= 4096 &&
              sizeof(UnitLaunch) <= 4096 && sizeof(AxpyLaunch) <= 4096 &&
              sizeof(ColStatLaunch) <= 4096 && sizeof(BnActLaunch) <= 4096 && sizeof(MaxPool3Launch) <= 4096 &&
              sizeof(BnApplyLaunch) <= 4096 && sizeof(TransposeLaunch) <= 4096 && sizeof(SgdLaunch) <= 4096,
              "kernel argument size");
int launch_conv(const ConvLaunch& L, int tiles, int dtype, int mode, int gk, int wn, int wm, hipStream_t s);
// wide 3x3 problems (k_gemm.hip): GEMM_BM x GEMM_BN tiles, bf16; the tile rows equal the tall conv
// tiles of 64-column problems, so BN partial rows do not depend on which kernel runs a problem
constexpr int GEMM_BM = 128, GEMM_BN = 128, GEMM_BK = 64;
constexpr int CONV_PRO_MAXC = 512;     // largest Cg of a forward BN prologue held in LDS
int launch_gemm(const ConvLaunch& L, int tiles, int mode, int tn, hipStream_t s);   // tn: 128 or 64
// the split problems' second pass: partial tiles summed in split order, then the epilogue, one
// workgroup per GEMM_RBN-column slab of a tile
int launch_gemm_reduce(const ConvLaunch& L, int tiles, int mode, hipStream_t s);
constexpr int GEMM_RBN = 16;
constexpr int GEMM_NARROW_MIN_TILES = 256;   // fewest tiles of a 64-column GEMM launch (else: halo kernel)
constexpr int GEMM_SPLIT_BELOW = 128;          // tiles of a problem below which its K is split
constexpr int GEMM_SPLIT_WG = 256;             // workgroups a split problem aims at (one per CU)
constexpr int GEMM_MAX_SPLIT = 16;
constexpr int GEMM_MIN_SPLIT_STEPS = 4;        // K steps of GEMM_BK per split, at least
// partial region of one chain: at most GEMM_SPLIT_WG partial tiles are live at once
constexpr size_t GEMM_KPART_BYTES = (size_t)GEMM_SPLIT_WG * GEMM_BM * GEMM_BN * 4;
// activation gather of wgrad_kernel: element-wise (any channel count), 16-byte chunks through the
// filter taps (Cg a multiple of the chunk), or pointwise (1x1 / stride 1 / pad 0: input row m)
enum { WG_GEN = 0, WG_VEC = 1, WG_PW = 2 };
int launch_wgrad(const WgradLaunch& L, int tiles, int dtype, int gather, hipStream_t s);
// wide 3x3 / stride 1 / pad 1 bf16 weight gradients (C_in, C_out multiples of 128) as 128 x 128 GEMM
// tiles over the pixels (k_gemm.hip); tiles_co = C_out / 128, tiles_k = 9 C_in / 128
int launch_wgrad_gemm(const WgradLaunch& L, int tiles, int tc, int tk, hipStream_t s);   // tc, tk: 128 or 64
// Streaming pointwise convolution of narrow problems (1x1 / stride 1 / pad 0, ncol % 32 != 0,
// K <= PW_MAXK): FWD with an optional BN prologue and EPI_STATS (no residual or addend); BWD with
// EPI_BN_MASK.  16-column workgroup tiles; wm = tiles of PW_TR rows per workgroup;
// tiles_m = ceil(M / (PW_TR wm)), tiles_n = ncol / 16.
int launch_pw(const ConvLaunch& L, int tiles, int dtype, int mode, hipStream_t s);
// BN backward sums of a 1x1 convolution's input BN (EPI_BN_MASK | EPI_NO_STORE problems):
// wm = tiles of BNSUM_TR rows per workgroup (bnsum_wm); tiles_m = ceil(M / (BNSUM_TR wm)),
// tiles_n = ceil(ncol / 64); K <= BNSUM_MAXK
int launch_bnsum(const ConvLaunch& L, int tiles, int dtype, hipStream_t s);
// 3x3 / stride 1 / pad 1 through an LDS halo tile: tiles_co = Co / 16, tiles_k = Cg / 16 blocks
int launch_wgrad3(const WgradLaunch& L, int tiles, int dtype, hipStream_t s);
int launch_colred(const ColRedLaunch& L, int tiles, hipStream_t s);
int launch_colstat(const ColStatLaunch& L, int tiles, int dtype, hipStream_t s);
// fused BN forward finalisation (bn_fwd_fuse): partial rows folded per group by its last workgroup
constexpr int BNF_GROUP = 32;
constexpr int BNF_STRIDE = 32;     // words between two counters (one 128-byte line each)
constexpr int BNF_MAX_ROWS = 512;  // producers with more partial rows keep the column-reduce pass
constexpr int BNF_MAX_WG = 512;    // ... and so do those of a level with more convolution workgroups
// counter words of a BN with C channels and at most `rows` partial rows: per column tile of >= 16
// columns, one counter per row group and one for the groups
__host__ __device__ inline long bnf_groups(long rows) { return rows / BNF_GROUP > 1 ? rows / BNF_GROUP : 1; }
inline long bnf_words(int C, long rows) {
  return (long)((C + 15) / 16) * (bnf_groups(rows < BNF_MAX_ROWS ? rows : BNF_MAX_ROWS) + 1) * BNF_STRIDE;
}
// zero-fill of word ranges (counters), one grouped launch
struct ZeroProb {
  unsigned* p;
  int words;
  int tile_begin;
};
struct ZeroLaunch {
  int tb[64];   // [0]: problem count; [p >= 1]: first workgroup of problem p (the lookup table)
  int n;
  ZeroProb p[64];
};
constexpr int ZERO_WORDS = 4096;   // words per workgroup
static_assert(sizeof(ZeroLaunch) <= 4096, "kernel argument size");
int launch_zero(const ZeroLaunch& L, int tiles, hipStream_t s);
int launch_bn_apply(const BnApplyLaunch& L, int tiles, int dtype, hipStream_t s);
int launch_bnact_fwd(const BnActLaunch& L, int tiles, int dtype, hipStream_t s);
int launch_bnact_bwd(const BnActLaunch& L, int tiles, int dtype, hipStream_t s);
int launch_maxpool3(const MaxPool3Launch& L, int tiles, int dtype, hipStream_t s);
int launch_transpose(const TransposeLaunch& L, int tiles, int dtype, hipStream_t s);
int launch_sub(const AxpyLaunch& L, int tiles, int dtype, hipStream_t s);
int launch_sumsq(const float* part, int n, float* out, hipStream_t s);
// shape of the head of a plan (batch, pixels and channels of ytilde, classes, storage type)
int head_geometry(const pnn_plan* p, int* B, int* HW, int* C, int* K, int* dtype);
int launch_head(const void* yt, const float* eps, const int32_t* labels, float* logits,
                float* loss, void* D_N, float* deps, float* scratch, int B, int HW, int C,
                int K, int dtype, unsigned* flag, hipStream_t s);

// tile sizes shared by host and device code
// conv workgroup tile: 16 x 16 sub-tiles per wave (row sub-tiles x column sub-tiles); a problem with
// ncol output columns takes wn = 4, 2 or 1 column sub-tiles and 64 x (CONV_SUBTILES / wn) rows of M
// (tall tiles) or 64 x conv_wm(wn, true) rows (short tiles)
constexpr int CONV_SUBTILES = 8;
inline int conv_wn(int ncol) { return (ncol % 64 == 0) ? 4 : (ncol % 32 == 0) ? 2 : 1; }
inline int conv_bm(int ncol) { return 64 * (CONV_SUBTILES / conv_wn(ncol)); }
// short tiles (single-problem launches such as the coarse chain's, which need more workgroups than
// tall tiles give): 2 sub-tiles per wave for 16- and 32-column tiles, 4 for 64-column tiles
inline int conv_wm(int wn, bool short_tiles) { return short_tiles ? (wn == 1 ? 2 : 1) : CONV_SUBTILES / wn; }
constexpr int SHORT_TILES_BELOW = 512;   // workgroups of a tall tiling below which short tiles pay
// row sub-tiles per wave of a k x k convolution problem with M rows and ncol columns in a segment
// that allows short tiles: short for 1x1 problems with few tall tiles (3x3 keep tall tiles)
inline int conv_rows_wm(int k, long M, int ncol, bool short_ok) {
  const int wn = conv_wn(ncol), tall = CONV_SUBTILES / wn;
  if (!short_ok || k != 1) return tall;
  const long tiles = (M + 64 * tall - 1) / (64 * tall) * (ncol / (16 * wn));
  return tiles < SHORT_TILES_BELOW ? conv_wm(wn, true) : tall;
}
constexpr int ELT_TILE = 2048;     // elements per workgroup of elementwise kernels
constexpr int SUB_TILE = 8192;     // elements per workgroup of the combine (sub_kernel)
constexpr int PNN_MAX_CHAINS = 4;  // streams the fine forward / backward may spread its segment groups over
constexpr int PW_TR = 64;          // rows per LDS tile of the streaming pointwise kernel
constexpr int PW_MAXK = 64;        // largest K of a streaming pointwise problem
constexpr int BNSUM_ROWS = 512;    // rows per BN-sum workgroup (short-tile segments: fewer, bnsum_wm)
constexpr int BNSUM_MAXK = 64;     // gradient channels of a BN-sum problem
constexpr int BNSUM_TR = 64;       // rows per LDS tile of bnsum_kernel
constexpr int COLSTAT_ROWS = 128;  // rows per column-statistics workgroup
constexpr int BNACT_PIX = 32;      // output pixels per bnact_bwd workgroup (one BN partial row)
constexpr int BNACT_MAXC = 512;    // channels of the chunked bnact path (per-channel constants in LDS)
// output pixels per bnact_fwd workgroup: about 1024 16-byte chunks of C channels, 1 to 64 pixels
// (channel counts off the chunk or above BNACT_MAXC: BNACT_PIX, the element-wise path)
inline int bnact_fwd_pix(int C, int es) {
  const int ve = 16 / es;
  if (C % ve != 0 || C > BNACT_MAXC) return BNACT_PIX;
  const int cc = C / ve;
  return 1024 / cc < 1 ? 1 : 1024 / cc > 64 ? 64 : 1024 / cc;
}
constexpr int CONV_HALO_BYTES = 40960;  // LDS of a 3x3 halo tile (input rows + halo, padded pixels)
// K steps whose filter fragments a wave keeps in registers, by column sub-tiles per wave (the
// register budget of narrow tiles, which carry more row sub-tiles, is smaller)
__host__ __device__ constexpr int conv_halo_nkb(int wn) { return wn == 1 ? 5 : wn == 2 ? 9 : 18; }
// unused 16-byte chunks after the cpp channel chunks of a halo pixel (output width Q): two for
// pixels of four or more chunks, a pixel stride of 8 dwords modulo 16 (measured: 8-wide maps with
// 64 channels took 4.3 LDS conflict cycles per LDS-active cycle with one chunk, 2.4 with two)
__host__ __device__ inline int conv_halo_pad(int cpp, int Q) { return cpp >= 4 ? 2 : 0; }


}  // namespace pnn
