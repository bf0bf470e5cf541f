// Resident forward of runs of pre-activation bottleneck residual units (Fig. ru: x_l = H_l(x_{l-1})
// + x_{l-1}; Table resnet, first stage: 32x32 maps, 64 channels squeezed to 16) for gfx950.
//
// One workgroup owns one image of one sub-network for the whole run of units:
//   * the residual stream x (1024 pixels x 64 channels, bf16) stays in registers from unit to unit,
//     in the layout an MFMA result has when its rows are channels and its columns pixels; read
//     with a matching permutation of the K index it is also the squeeze's A operand, so no
//     transpose is ever needed;
//   * the squeeze output z1 and the 3x3 output z2 (1024 x 16 each) live in one LDS buffer with a
//     zero border of one pixel (the 3x3's zero padding), activated in place once their batch
//     statistics are known.
// Batch normalisation needs statistics over the whole batch, so every BN point is a grid-wide
// barrier: each workgroup writes its image's per-channel (mean, sum of squared deviations), all
// workgroups of the sub-network then combine the batch's partials in the same fixed order (fp64),
// and apply them.  Three barriers per unit.  HBM traffic per unit and image: the stored z1, z2 and
// unit output (what the backward reads), about 192 KB, against about 512 KB for the same unit run
// layer by layer.
//
// Every workgroup of a launch must be resident at once: the host sizes launches from the occupancy
// (sub-networks in waves of at most that many images, one launch at a time on one stream), and every
// barrier wait is bounded: after UNIT_SPIN_LIMIT polls it sets an error flag and stops waiting (and
// later barriers no longer wait), so a launch always ends.
#include "device_common.h"
#include "pnn_internal.h"

namespace pnn {

namespace {

constexpr int UH = UNIT_H, UW = UNIT_W, UC = UNIT_C, UM = UNIT_MID;
constexpr int UPX = UH * UW;          // pixels per image
constexpr int UPB = UPX / 16;         // 16-pixel blocks per image
constexpr int UWV = UNIT_WAVES;       // waves per workgroup
constexpr int UNT = 64 * UWV;         // threads per workgroup
constexpr int UBW = UPB / UWV;        // blocks per wave
constexpr int UCB = UC / 16;          // 16-channel blocks of x
constexpr int ZPW = UW + 2;           // padded row
constexpr int ZPIX = (UH + 2) * ZPW;  // padded pixels
constexpr unsigned UNIT_SPIN_LIMIT = 1u << 21;

static_assert(UM == 16 && UC % 32 == 0 && UPB % UWV == 0 && UW % 16 == 0 && UNT % UC == 0 &&
              UPX % (UNT / 16) == 0, "unit kernel layout");

__device__ __forceinline__ int padpix(int px) { return (px / UW + 1) * ZPW + px % UW + 1; }

// A zero the optimiser cannot see through: adding it to a per-lane base inside the unit loop keeps
// the many addresses derived from that base (one per unrolled block) from being hoisted out of the
// loop, where they would occupy registers for the whole kernel; inside, each folds into an
// instruction's immediate offset.
__device__ __forceinline__ int opaque_zero() {
  int z = 0;
  asm volatile("" : "+v"(z));
  return z;
}

// Padded LDS pixel of block p's pixel 16 P + c (P = UBW wave + p, c < 16) relative to the lane's
// base ((UBW / 2) wave + 1) ZPW + 1: blocks come in pairs per image row.
__device__ __forceinline__ constexpr int blk_off(int p, int c) { return (p / 2) * ZPW + (p % 2) * 16 + c; }

// Barrier of the nwg workgroups of one job: job words arrive (arrivals) and gen (generation), on
// cache lines of their own; glob[0] is the launch's error flag, glob[1] counts completed barriers.
// What workgroups exchange across it (the BN partials) is written and read with device-coherent
// accesses, so no cache-wide fence is needed (a device-scope fence writes back and invalidates the
// whole L2 of the XCD): every wave waits for its own stores, then one thread arrives and waits.
__device__ void job_sync(unsigned* arrive, unsigned* gen, unsigned* glob, unsigned nwg) {
  wait_mem();
  __syncthreads();
  if (threadIdx.x == 0) {
    if (__hip_atomic_load(glob, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
      const unsigned g = __hip_atomic_load(gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      wait_mem();                      // the generation read before the arrival
      const unsigned old = __hip_atomic_fetch_add(arrive, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (old == nwg - 1) {
        __hip_atomic_store(arrive, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        wait_mem();                    // the reset lands before the next generation opens
        __hip_atomic_fetch_add(gen, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_fetch_add(glob + 1, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      } else {
        unsigned spins = 0;
        while (__hip_atomic_load(gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == g) {
          __builtin_amdgcn_s_sleep(2);
          if (++spins > UNIT_SPIN_LIMIT) {
            __hip_atomic_store(glob, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            break;
          }
        }
      }
    }
  }
  __syncthreads();
}

__device__ __forceinline__ float relu_bn(float v, float sc, float sh) { return fmaxf(fmaf(v, sc, sh), 0.0f); }

// The residual stream's packed bf16 pair, made opaque to the optimiser at each use: the compiler
// would otherwise keep all of x unpacked to fp32 (twice the registers) across the units.
__device__ __forceinline__ uint2 packed(uint2 v) {
  asm volatile("" : "+v"(v.x), "+v"(v.y));
  return v;
}
__device__ __forceinline__ float bf_elem(uint2 v, int i) {
  const uint32_t w = i < 2 ? v.x : v.y;
  return __uint_as_float(i & 1 ? (w & 0xffff0000u) : (w << 16));
}

// Per-channel (mean, sum of squared deviations) of the image's 16-channel buffer in LDS (interior
// pixels), two passes; thread t < 16 writes channel t's pair to part.
__device__ void image_stats16(const uint16_t* zs, float* red, float* part) {
  constexpr int NG = UNT / 16, GP = UPX / NG;          // pixel groups, pixels per group
  const int t = threadIdx.x, o = t & 15, q = t >> 4;
  float s = 0.f;
  for (int px = q * GP; px < (q + 1) * GP; ++px) s += bf2f(zs[padpix(px) * 16 + o]);
  red[t] = s;
  __syncthreads();
  if (t < 16) {
    float a = 0.f;
    for (int k = 0; k < NG; ++k) a += red[k * 16 + t];
    red[UNT + t] = a / (float)UPX;
  }
  __syncthreads();
  const float mean = red[UNT + o];
  float m2 = 0.f;
  for (int px = q * GP; px < (q + 1) * GP; ++px) {
    const float d = bf2f(zs[padpix(px) * 16 + o]) - mean;
    m2 += d * d;
  }
  red[t] = m2;
  __syncthreads();
  if (t < 16) {
    float a = 0.f;
    for (int k = 0; k < NG; ++k) a += red[k * 16 + t];
    st_coherent((float2*)part + t, make_float2(red[UNT + t], a));
  }
  __syncthreads();
}

// BN statistics of C channels from the batch's per-image partials part[B][C] (mean, M2 over UPX
// pixels each), fp64 in a fixed order (identical in every workgroup): scale / shift to sc / sh
// (LDS), and mean / invstd / scale / shift to stats when stats != nullptr.
template <int C>
__device__ void batch_stats(const float* part, int B, const float* gamma_beta, float* stats, double* dred,
                            float* sc, float* sh) {
  constexpr int NQ = UNT / C;
  constexpr int U = 128 / NQ < 1 ? 1 : 128 / NQ > 16 ? 16 : 128 / NQ;   // loads in flight per thread
  const int t = threadIdx.x, c = t % C, q = t / C;
  double a = 0.0, qq = 0.0;
  for (int n0 = q; n0 < B; n0 += U * NQ) {
    float2 v[U];
#pragma unroll
    for (int k = 0; k < U; ++k)
      v[k] = n0 + k * NQ < B ? ld_coherent((const float2*)part + (long)(n0 + k * NQ) * C + c) : make_float2(0.f, 0.f);
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const double m = (double)v[k].x;
      a += (double)UPX * m;
      qq += (double)v[k].y + (double)UPX * m * m;
    }
  }
  dred[t] = a;
  dred[UNT + t] = qq;
  __syncthreads();
  if (t < C) {
    double A = 0.0, Q = 0.0;
    for (int k = 0; k < NQ; ++k) {
      A += dred[k * C + t];
      Q += dred[UNT + k * C + t];
    }
    const double M = (double)B * UPX;
    const double mean = A / M;
    double var = Q / M - mean * mean;
    if (var < 0.0) var = 0.0;
    const float invstd = (float)(1.0 / sqrt(var + (double)PNN_BN_EPS));
    const float scale = gamma_beta[t] * invstd;
    const float shift = gamma_beta[C + t] - (float)mean * scale;
    sc[t] = scale;
    sh[t] = shift;
    if (stats != nullptr) {
      stats[t] = (float)mean;
      stats[C + t] = invstd;
      stats[2 * C + t] = scale;
      stats[3 * C + t] = shift;
    }
  }
  __syncthreads();
}

}  // namespace

__global__ void unit_sync_reset_kernel(unsigned* sync) {
  const int t = threadIdx.x;
  if (t < 2) sync[t] = 0u;
  else if (t < 2 + 2 * UNIT_MAXJ) sync[unit_sync_word(t / 2 - 1, t % 2)] = 0u;
}

__global__ __launch_bounds__(UNT) void unit_fwd_kernel(const UnitLaunch L) {
  __shared__ __attribute__((aligned(16))) uint16_t zs[ZPIX * 16];
  __shared__ __attribute__((aligned(16))) float red[UNT + 64];
  __shared__ double dred[2 * UNT];
  __shared__ float sc1[UC], sh1[UC], sc2[UM], sh2[UM];

  int ji = 0;
  while (ji + 1 < L.n && (int)blockIdx.x >= L.j[ji + 1].wg_begin) ++ji;
  const UnitJob& J = L.j[ji];
  const int n = blockIdx.x - J.wg_begin;               // image
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63, r16 = lane & 15, g = lane >> 4;

  for (int i = tid; i < ZPIX * 16 / 8; i += UNT) ((uint4*)zs)[i] = make_uint4(0, 0, 0, 0);

  // x of the first unit: lane (g, r16) of wave w holds, for each of its blocks p and channel block
  // b, channels 16 b + 4 g + i (i < 4) of pixel 16 (UBW w + p) + r16
  uint2 xr[UBW][UCB];
  {
    const uint16_t* xin = (const uint16_t*)J.x_in + (long)n * UPX * UC + (16 * UBW * wave + r16) * UC + 4 * g;
#pragma unroll
    for (int p = 0; p < UBW; ++p)
#pragma unroll
      for (int b = 0; b < UCB; ++b) xr[p][b] = *(const uint2*)(xin + 16 * p * UC + 16 * b);
  }
  // BN(x) of the first unit: scale / shift from the saved statistics
  if (tid < UC) {
    const float* st = (const float*)(J.saved + J.s1);
    sc1[tid] = st[2 * UC + tid];
    sh1[tid] = st[3 * UC + tid];
  }
  __syncthreads();

  float* part_z1 = J.part;
  float* part_z2 = J.part + (long)L.B * UM * 2;
  float* part_x = J.part + (long)2 * L.B * UM * 2;

  unsigned* const arrive = L.sync + unit_sync_word(ji, 0);
  unsigned* const gen = L.sync + unit_sync_word(ji, 1);
  for (int u = 0; u < J.nu; ++u) {
    // per-lane LDS bases of this unit (see opaque_zero): lane pixel row base of the squeeze / z2
    // writes (pixels 4 g + i of a block), and of the 3x3 / expand reads (pixel r16 of a block)
    const int oz = opaque_zero();
    uint16_t* zw = zs + (((UBW / 2) * wave + 1) * ZPW + 1 + 4 * g + oz) * 16 + r16;
    const uint16_t* zr = zs + (((UBW / 2) * wave + 1) * ZPW + 1 + r16 + oz) * 16;
    const bool last = u == J.nu - 1;
    const char* prm = J.params;
    const unsigned w1 = J.w1 + u * L.dw, w2 = J.w2 + u * L.dw, w3 = J.w3 + u * L.dw;
    const unsigned gb2 = J.g2 + u * L.dg, gb3 = J.g3 + u * L.dg;

    // ---- squeeze: z1[px][o] = sum_k ReLU(BN(x))[px][k] W1[o][k], K in the permuted order of x ----
    {
      bf16x8 wf[UC / 32];
#pragma unroll
      for (int s = 0; s < UC / 32; ++s) {
        const uint16_t* w = (const uint16_t*)(prm + w1) + r16 * UC + 32 * s + 4 * g;
        const uint2 lo = *(const uint2*)w, hi = *(const uint2*)(w + 16);
        wf[s] = __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
      }
      float sc[UCB][4], sh[UCB][4];
#pragma unroll
      for (int b = 0; b < UCB; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          sc[b][i] = sc1[16 * b + 4 * g + i];
          sh[b][i] = sh1[16 * b + 4 * g + i];
        }
#pragma unroll
      for (int p = 0; p < UBW; ++p) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < UC / 32; ++s) {
          bf16x8 a;
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const uint2 v = packed(xr[p][2 * s + h]);
#pragma unroll
            for (int i = 0; i < 4; ++i) a[4 * h + i] = (__bf16)relu_bn(bf_elem(v, i), sc[2 * s + h][i], sh[2 * s + h][i]);
          }
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, wf[s], acc, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < 4; ++i) zw[blk_off(p, i) * 16] = f2bf(acc[i]);
        __builtin_amdgcn_sched_barrier(0);     // one block at a time: short live ranges
      }
    }
    __syncthreads();
    {
      image_stats16(zs, red, part_z1 + (long)n * UM * 2);
      uint16_t* z1g = (uint16_t*)(J.saved + J.z1 + (long)u * L.dz) + (long)n * UPX * UM;
      for (int k = tid; k < UPX * 2; k += UNT)
        *(uint4*)(z1g + k * 8) = *(const uint4*)(zs + padpix(k >> 1) * 16 + (k & 1) * 8);
    }
    job_sync(arrive, gen, L.sync, L.B);

    // ---- BN(z1), then the 3x3 on the activated buffer ----
    {
      batch_stats<UM>(part_z1, L.B, (const float*)(prm + gb2), n == 0 ? (float*)(J.saved + J.s2 + u * L.ds) : nullptr,
                      dred, sc2, sh2);
      for (int k = tid; k < UPX * 2; k += UNT) {
        uint4* q = (uint4*)(zs + padpix(k >> 1) * 16 + (k & 1) * 8);
        Chunk<uint16_t> c;
        unpack_chunk<uint16_t>(*q, c);
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = relu_bn(c.v[e], sc2[(k & 1) * 8 + e], sh2[(k & 1) * 8 + e]);
        store_chunk<uint16_t>(q, 0, v);
      }
    }
    __syncthreads();
    uint2 z2r[UBW];
    {
      // K step s: lane groups 0, 1 take tap 2 s (channels 0-7, 8-15), groups 2, 3 tap 2 s + 1
      bf16x8 wf[5];
#pragma unroll
      for (int s = 0; s < 5; ++s) {
        const int tap = 2 * s + (g >> 1);
        wf[s] = tap < 9 ? __builtin_bit_cast(bf16x8, *(const uint4*)((const uint16_t*)(prm + w2) + r16 * 144 + tap * 16 + (g & 1) * 8))
                        : __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
      }
#pragma unroll
      for (int p = 0; p < UBW; ++p) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < 5; ++s) {
          // lane groups 0, 1 read tap 2 s, groups 2, 3 tap 2 s + 1 (the last K step's upper half
          // is zero)
          uint4 raw = make_uint4(0, 0, 0, 0);
          const int ta = 2 * s, tb = 2 * s + 1;
          const int oa = ((ta / 3 - 1) * ZPW + ta % 3 - 1) * 16, ob = ((tb / 3 - 1) * ZPW + tb % 3 - 1) * 16;
          if (g < 2) raw = *(const uint4*)(zr + blk_off(p, 0) * 16 + oa + g * 8);
          else if (tb < 9) raw = *(const uint4*)(zr + blk_off(p, 0) * 16 + ob + (g - 2) * 8);
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, raw), wf[s], acc, 0, 0, 0);
        }
        z2r[p] = make_uint2((uint32_t)f2bf(acc[0]) | ((uint32_t)f2bf(acc[1]) << 16),
                            (uint32_t)f2bf(acc[2]) | ((uint32_t)f2bf(acc[3]) << 16));
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    __syncthreads();
    {
#pragma unroll
      for (int p = 0; p < UBW; ++p) {
        zw[blk_off(p, 0) * 16] = (uint16_t)(z2r[p].x & 0xffff);
        zw[blk_off(p, 1) * 16] = (uint16_t)(z2r[p].x >> 16);
        zw[blk_off(p, 2) * 16] = (uint16_t)(z2r[p].y & 0xffff);
        zw[blk_off(p, 3) * 16] = (uint16_t)(z2r[p].y >> 16);
      }
    }
    __syncthreads();
    {
      image_stats16(zs, red, part_z2 + (long)n * UM * 2);
      uint16_t* z2g = (uint16_t*)(J.saved + J.z2 + (long)u * L.dz) + (long)n * UPX * UM;
      for (int k = tid; k < UPX * 2; k += UNT)
        *(uint4*)(z2g + k * 8) = *(const uint4*)(zs + padpix(k >> 1) * 16 + (k & 1) * 8);
    }
    job_sync(arrive, gen, L.sync, L.B);

    // ---- BN(z2), then the expand 1x1 with the residual: x' = W3 ReLU(BN(z2)) + x ----
    const bool xbn = !last || J.sN != 0xffffffffu;   // x' is normalised by a BN
    {
      batch_stats<UM>(part_z2, L.B, (const float*)(prm + gb3), n == 0 ? (float*)(J.saved + J.s3 + u * L.ds) : nullptr,
                      dred, sc2, sh2);
      for (int k = tid; k < UPX * 2; k += UNT) {
        uint4* q = (uint4*)(zs + padpix(k >> 1) * 16 + (k & 1) * 8);
        Chunk<uint16_t> c;
        unpack_chunk<uint16_t>(*q, c);
        float v[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = relu_bn(c.v[e], sc2[(k & 1) * 8 + e], sh2[(k & 1) * 8 + e]);
        store_chunk<uint16_t>(q, 0, v);
      }
    }
    __syncthreads();
    {
      bf16x8 wf[UCB];
#pragma unroll
      for (int b = 0; b < UCB; ++b)
        wf[b] = g < 2 ? __builtin_bit_cast(bf16x8, *(const uint4*)((const uint16_t*)(prm + w3) + (16 * b + r16) * UM + 8 * g))
                      : __builtin_bit_cast(bf16x8, make_uint4(0, 0, 0, 0));
      float s1[UCB][4];
#pragma unroll
      for (int b = 0; b < UCB; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i) s1[b][i] = 0.f;
      uint16_t* xo = last && J.sN == 0xffffffffu && J.y_out != nullptr
                         ? (uint16_t*)J.y_out
                         : (uint16_t*)(J.saved + J.xo + (long)u * L.dz);
      xo += (long)n * UPX * UC + (16 * UBW * wave + r16) * UC + 4 * g + oz;
#pragma unroll
      for (int p = 0; p < UBW; ++p) {
        const uint4 raw = g < 2 ? *(const uint4*)(zr + blk_off(p, 0) * 16 + 8 * g) : make_uint4(0, 0, 0, 0);
        const bf16x8 bv = __builtin_bit_cast(bf16x8, raw);
#pragma unroll
        for (int b = 0; b < UCB; ++b) {
          f32x4 acc = {0.f, 0.f, 0.f, 0.f};
          acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[b], bv, acc, 0, 0, 0);
          const uint2 v = packed(xr[p][b]);
          float o[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            o[i] = bf2f(f2bf(acc[i] + bf_elem(v, i)));
            s1[b][i] += o[i];
          }
          xr[p][b] = make_uint2((uint32_t)f2bf(o[0]) | ((uint32_t)f2bf(o[1]) << 16),
                                (uint32_t)f2bf(o[2]) | ((uint32_t)f2bf(o[3]) << 16));
          *(uint2*)(xo + 16 * p * UC + 16 * b) = xr[p][b];
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      if (xbn) {
        // per-channel mean over the image: lanes with the same g hold the same channels
#pragma unroll
        for (int b = 0; b < UCB; ++b)
#pragma unroll
          for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int o = 1; o < 16; o <<= 1) s1[b][i] += __shfl_xor(s1[b][i], o, 64);
        if (r16 == 0)
#pragma unroll
          for (int b = 0; b < UCB; ++b)
#pragma unroll
            for (int i = 0; i < 4; ++i) red[wave * UC + 16 * b + 4 * g + i] = s1[b][i];
      }
    }
    __syncthreads();
    if (xbn && tid < UC) {
      float a = 0.f;
      for (int w = 0; w < UWV; ++w) a += red[w * UC + tid];
      red[UNT + tid] = a / (float)UPX;
    }
    __syncthreads();
    if (xbn) {
      float s2[UCB][4];
#pragma unroll
      for (int b = 0; b < UCB; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i) s2[b][i] = 0.f;
#pragma unroll
      for (int p = 0; p < UBW; ++p)
#pragma unroll
        for (int b = 0; b < UCB; ++b) {
          const uint2 v = packed(xr[p][b]);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float d = bf_elem(v, i) - red[UNT + 16 * b + 4 * g + i];
            s2[b][i] += d * d;
          }
          __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
      for (int b = 0; b < UCB; ++b)
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int o = 1; o < 16; o <<= 1) s2[b][i] += __shfl_xor(s2[b][i], o, 64);
      __syncthreads();
      if (r16 == 0)
#pragma unroll
        for (int b = 0; b < UCB; ++b)
#pragma unroll
          for (int i = 0; i < 4; ++i) red[wave * UC + 16 * b + 4 * g + i] = s2[b][i];
      __syncthreads();
      if (tid < UC) {
        float a = 0.f;
        for (int w = 0; w < UWV; ++w) a += red[w * UC + tid];
        st_coherent((float2*)part_x + (long)n * UC + tid, make_float2(red[UNT + tid], a));
      }
    }
    job_sync(arrive, gen, L.sync, L.B);

    // ---- BN(x') for the next unit ----
    if (xbn) {
      const unsigned gn = last ? J.gN : J.g1 + (u + 1) * L.dg;
      const unsigned sn = last ? J.sN : J.s1 + (u + 1) * L.ds;
      batch_stats<UC>(part_x, L.B, (const float*)(prm + gn), n == 0 ? (float*)(J.saved + sn) : nullptr, dred,
                      sc1, sh1);
    }
  }
}

int launch_unit_reset(unsigned* sync, hipStream_t s) {
  hipLaunchKernelGGL(unit_sync_reset_kernel, dim3(1), dim3(64), 0, s, sync);
  return (int)hipGetLastError();
}

int launch_unit_fwd(const UnitLaunch& L, hipStream_t s) {
  hipLaunchKernelGGL(unit_fwd_kernel, dim3(L.nwg), dim3(UNT), 0, s, L);
  return (int)hipGetLastError();
}

int unit_fwd_occupancy() {
  int blocks = 0, dev = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, unit_fwd_kernel, UNT, 0) != hipSuccess) return 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return blocks * cus;
}

}  // namespace pnn
