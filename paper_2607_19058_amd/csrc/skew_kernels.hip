// skew_kernels.hip -- gfx950 kernels of one SkewAdam step (Sec. 3, Eq. 1, Alg. 1).
//
// A step is four stream-ordered launches over device-resident work-item tables;
// each launch covers every tensor of the table (e.g. all experts of a layer):
//   p1    factored tensors: per tile, partial row and column sums of g^2 (Eq. 1)
//   fold  factored tensors: R, C EMA (Eq. 1), 1/sqrt(R_i), sums of R for mean(R)
//   p2    every tensor: per tile, sum of squares of the unclipped update (Alg. 1)
//   p3    every tensor: clip factor, momentum / exact-v update, weight update,
//         dithered bf16 write-back (Sec. 3 "Update clipping and low-precision updates")
// Reductions are deterministic (fixed-order partials; no float atomics), so two
// runs on the same inputs produce identical bits.
//
// Tile: tr rows x (512*cw) columns. A work-group is 4 wave64; wave w takes rows
// r0+w, r0+w+4, ...; lane l covers 8 consecutive columns (one 16-byte bf16 load)
// in each 512-column chunk.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "skew_internal.h"

namespace skew {
namespace {

// Tensor pointers come from the device-resident table, so the compiler cannot infer
// their address space; these accessors make every data access a global (not flat) one.
template <class T>
__device__ __forceinline__ T ldg(const T *p) {
  return *(const __attribute__((address_space(1))) T *)p;
}
template <class T>
__device__ __forceinline__ void stg(T *p, T v) {
  *(__attribute__((address_space(1))) T *)p = v;
}
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint4 ldg(const uint4 *p) {
  const u32x4_t v = ldg(reinterpret_cast<const u32x4_t *>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float4 ldg(const float4 *p) {
  const f32x4_t v = ldg(reinterpret_cast<const f32x4_t *>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void stg(uint4 *p, uint4 v) {
  const u32x4_t u = {v.x, v.y, v.z, v.w};
  stg(reinterpret_cast<u32x4_t *>(p), u);
}
__device__ __forceinline__ void stg(float4 *p, float4 v) {
  const f32x4_t u = {v.x, v.y, v.z, v.w};
  stg(reinterpret_cast<f32x4_t *>(p), u);
}

__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }
__device__ __forceinline__ float bf_one(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// max(a, b) that returns `a` when it is NaN (b is a finite constant): NaN propagates.
__device__ __forceinline__ float max_nan(float a, float b) { return (a < b) ? b : a; }

__device__ __forceinline__ void unpack8(const uint4 &u, float *o) {
  o[0] = bf_lo(u.x); o[1] = bf_hi(u.x);
  o[2] = bf_lo(u.y); o[3] = bf_hi(u.y);
  o[4] = bf_lo(u.z); o[5] = bf_hi(u.z);
  o[6] = bf_lo(u.w); o[7] = bf_hi(u.w);
}

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// two floats -> two bf16, round to nearest even, packed low|high
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  f32x2 v = {a, b};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}
__device__ __forceinline__ uint16_t to_bf16(float a) { return __builtin_bit_cast(uint16_t, (__bf16)a); }

// SplitMix64 output function (Steele, Lea, Flood, OOPSLA 2014).
__device__ __forceinline__ uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
// MurmurHash3 32-bit finalizer (public domain).
__device__ __forceinline__ uint32_t fmix32(uint32_t h) {
  h ^= h >> 16;
  h *= 0x85EBCA6Bu;
  h ^= h >> 13;
  h *= 0xC2B2AE35u;
  h ^= h >> 16;
  return h;
}

// Counter-based dither source: one 32-bit hash per element pair p = idx >> 1,
// keyed by (seed, step, tensor id). Element 2p takes the low 16 bits, 2p+1 the high.
struct Dither {
  uint32_t klo, khi, inner0;
  __device__ __forceinline__ Dither(uint64_t seed, int64_t step, uint64_t id) {
    const uint64_t k = mix64(mix64(mix64(seed) ^ (uint64_t)step) ^ id);
    klo = (uint32_t)k;
    khi = (uint32_t)(k >> 32);
    inner0 = fmix32(khi);
  }
  __device__ __forceinline__ uint32_t pair(uint64_t p) const {
    const uint32_t ph = (uint32_t)(p >> 32);
    const uint32_t inner = (ph == 0u) ? inner0 : fmix32(ph ^ khi);
    return fmix32((uint32_t)p ^ klo ^ inner);
  }
};

// e * 2^-24 with e = 2*u16 + 1 - 2^16, for u16 = bits 7..22 of `field`:
// the float 2^-7 (1 + (2 u16 + 1) 2^-17) minus 1.5 * 2^-7, both steps exact.
__device__ __forceinline__ float dither_lo(uint32_t h) {
  return __uint_as_float(0x3C000040u | ((h << 7) & 0x7FFF80u)) - 0.01171875f;
}
__device__ __forceinline__ float dither_hi(uint32_t h) {
  return __uint_as_float(0x3C000040u | ((h >> 9) & 0x7FFF80u)) - 0.01171875f;
}
__device__ __forceinline__ float dither_of(uint32_t h, uint64_t idx) { return (idx & 1u) ? dither_hi(h) : dither_lo(h); }

// fixed-order tree over the work-group (every thread gets the total)
__device__ __forceinline__ double block_sum(double x, double *sh) {
  sh[threadIdx.x] = x;
  __syncthreads();
#pragma unroll
  for (int s = kThreads / 2; s > 0; s >>= 1) {
    if ((int)threadIdx.x < s) sh[threadIdx.x] += sh[threadIdx.x + s];
    __syncthreads();
  }
  const double r = sh[0];
  __syncthreads();
  return r;
}

// A tile is one row band (rows band, band + ntr, band + 2 ntr, ...: interleaved, so that
// the work-groups running at the same time on one tensor read neighbouring rows) times
// one column strip of 512*cw columns.
struct Tile {
  int64_t nr, c0, stride;   // local rows, first column, row stride between local rows
  int band, strip;
  __device__ __forceinline__ int64_t row(int64_t lr) const { return band + lr * stride; }
};
__device__ __forceinline__ Tile tile_of(const DevTensor &t, int tile) {
  Tile g;
  g.band = tile / t.ntc;
  g.strip = tile - g.band * t.ntc;
  g.stride = t.ntr;
  g.nr = (t.n - g.band + t.ntr - 1) / t.ntr;
  g.c0 = (int64_t)g.strip * kChunk * t.cw;
  return g;
}

// Wave -> (chunk, row) map inside a tile: the cw chunks of a row go to cw adjacent waves,
// so one work-group iteration reads kWaves / cw whole tile rows (up to 4 KB contiguous),
// and every wave keeps the same 512 columns for the whole tile.
struct WaveMap {
  int wq, wr, rpi, lane;
  int64_t col;   // first of the lane's 8 columns
  __device__ __forceinline__ WaveMap(const DevTensor &t, const Tile &tl) {
    const int wave = threadIdx.x >> 6;
    lane = threadIdx.x & 63;
    wq = wave % t.cw;
    wr = wave / t.cw;
    rpi = kWaves / t.cw;
    col = tl.c0 + (int64_t)wq * kChunk + lane * 8;
  }
};

__device__ __forceinline__ void load_g8(const DevTensor &t, int64_t i, int64_t col, float *g) {
  const uint16_t *row = t.g + i * t.ld;
  if (t.vec) {
    if (col < t.m) {
      unpack8(ldg(reinterpret_cast<const uint4 *>(row + col)), g);
    } else {
#pragma unroll
      for (int e = 0; e < 8; e++) g[e] = 0.f;
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; e++) g[e] = (col + e < t.m) ? bf_one(ldg(row + col + e)) : 0.f;
  }
}

// --------------------------------------------------------------------------------------------
// p1: partial row / column sums of g^2 (Eq. 1: mean_c and mean_r of G (.) G).
// Squares of bf16 values are exact in double and the sums stay far from double
// rounding, so every partial is (nearly) the exact sum, independent of order.
// --------------------------------------------------------------------------------------------
__device__ __forceinline__ double wave_sum_d(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}

constexpr int kRowSlots = (int)(kTileElems / kChunk);   // tile rows x chunks per row

__global__ __launch_bounds__(kThreads) void p1_kernel(const DevTensor *__restrict__ TT,
                                                      const Item *__restrict__ items) {
  __shared__ double colsh[kWaves][kChunk];
  __shared__ double rowsh[kRowSlots];
  const Item it = items[blockIdx.x];
  const DevTensor &t = TT[it.tensor];
  const Tile tl = tile_of(t, it.tile);
  const WaveMap wm(t, tl);
  const int cw = t.cw;

  double acc[8];
#pragma unroll
  for (int e = 0; e < 8; e++) acc[e] = 0.0;
  for (int64_t lr = wm.wr; lr < tl.nr; lr += 2 * wm.rpi) {
    const bool two = lr + wm.rpi < tl.nr;
    float ga[8], gb[8];
    load_g8(t, tl.row(lr), wm.col, ga);
    if (two) load_g8(t, tl.row(lr + wm.rpi), wm.col, gb);
    double ra = 0.0, rb = 0.0;
#pragma unroll
    for (int e = 0; e < 8; e++) {
      const double x = (double)ga[e];
      ra = fma(x, x, ra);
      acc[e] = fma(x, x, acc[e]);
    }
    if (two) {
#pragma unroll
      for (int e = 0; e < 8; e++) {
        const double x = (double)gb[e];
        rb = fma(x, x, rb);
        acc[e] = fma(x, x, acc[e]);
      }
    }
    ra = wave_sum_d(ra);
    rb = wave_sum_d(rb);
    if (wm.lane == 0) {
      rowsh[lr * cw + wm.wq] = ra;
      if (two) rowsh[(lr + wm.rpi) * cw + wm.wq] = rb;
    }
  }
#pragma unroll
  for (int e = 0; e < 8; e++) colsh[threadIdx.x >> 6][wm.lane * 8 + e] = acc[e];
  __syncthreads();
  for (int r = threadIdx.x; r < (int)tl.nr; r += kThreads) {
    double s = 0.0;
    for (int q = 0; q < cw; q++) s += rowsh[r * cw + q];
    stg(t.rowpart + (int64_t)tl.strip * t.n + tl.row(r), s);
  }
  for (int c = threadIdx.x; c < kChunk * cw; c += kThreads) {
    const int q = c / kChunk, cc = c - q * kChunk;
    double s = 0.0;
    for (int w = q; w < kWaves; w += cw) s += colsh[w][cc];
    const int64_t col = tl.c0 + c;
    if (col < t.m) stg(t.colpart + (int64_t)tl.band * t.m + col, s);
  }
}

// --------------------------------------------------------------------------------------------
// fold: R_i <- b2 R_i + a2 r_i, C_j <- b2 C_j + a2 c_j (Eq. 1), 1/sqrt(R_i), sums of R
// --------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void fold_kernel(const DevTensor *__restrict__ TT,
                                                        const Item *__restrict__ items, StepConsts k) {
  __shared__ double sh[kThreads];
  const Item it = items[blockIdx.x];
  const DevTensor &t = TT[it.tensor];
  if (it.tile < t.nfr) {
    const int64_t i = (int64_t)it.tile * kFold + threadIdx.x;
    double rn = 0.0;
    if (i < t.n) {
      double s = 0.0;
      for (int q = 0; q < t.ntc; q++) s += ldg(t.rowpart + (int64_t)q * t.n + i);
      const float ri = (float)(s / (double)t.m);
      const float R = fmaf(k.a2, ri, __fmul_rn(k.b2, ldg(t.R + i)));
      stg(t.R + i, R);
      stg(t.ainv + i, 1.0 / sqrt((double)R));
      rn = (double)R;
    }
    const double tot = block_sum(rn, sh);
    if (threadIdx.x == 0) stg(t.rsum + it.tile, tot);
  } else {
    const int64_t j = (int64_t)(it.tile - t.nfr) * kFold + threadIdx.x;
    if (j < t.m) {
      double s = 0.0;
      for (int b = 0; b < t.ntr; b++) s += ldg(t.colpart + (int64_t)b * t.m + j);
      const float cj = (float)(s / (double)t.n);
      stg(t.C + j, fmaf(k.a2, cj, __fmul_rn(k.b2, ldg(t.C + j))));
    }
  }
}

// Column factors of the rank-one reconstruction: q = max(mean R, eps) and c'_j = C_j / q
// rounded as the oracle rounds them; b_j = 1/sqrt(c'_j) in double, so that
// 1/D_ij = min(b_j / sqrt(R_i), 1/sqrt(eps)) (Eq. 1 reconstruction with the Alg. 1 clamps).
// fixed-order work-group sum of p[0..n): thread j sums p[j], p[j + 256], ..., then a tree;
// every thread of the work-group must call it
__device__ __forceinline__ double wg_sum(const double *p, int64_t n, double *sh) {
  double s = 0.0;
  for (int64_t c = threadIdx.x; c < n; c += kThreads) s += ldg(p + c);
  return block_sum(s, sh);
}
// q = max(mean R, eps) for a factored tensor (the clamp of the reconstruction)
__device__ __forceinline__ float mean_r_clamped(const DevTensor &t, float eps, double *sh) {
  return max_nan((float)(wg_sum(t.rsum, t.nfr, sh) / (double)t.n), eps);
}
__device__ __forceinline__ double col_factor(const DevTensor &t, int64_t col, float q) {
  return 1.0 / sqrt((double)(ldg(t.C + col) / q));
}

// 8 momentum values at a 32-byte aligned position
__device__ __forceinline__ void load_m8(const float *p, float *o) {
  const float4 a = ldg(reinterpret_cast<const float4 *>(p));
  const float4 b = ldg(reinterpret_cast<const float4 *>(p + 4));
  o[0] = a.x; o[1] = a.y; o[2] = a.z; o[3] = a.w; o[4] = b.x; o[5] = b.y; o[6] = b.z; o[7] = b.w;
}
__device__ __forceinline__ void store_m8(float *p, const float *v) {
  stg(reinterpret_cast<float4 *>(p), make_float4(v[0], v[1], v[2], v[3]));
  stg(reinterpret_cast<float4 *>(p + 4), make_float4(v[4], v[5], v[6], v[7]));
}

// --------------------------------------------------------------------------------------------
// p2: per-tile sum of squares of the unclipped update U_hat (Alg. 1, before clipping).
//
// The clip factor must round to the oracle's float, so the sum must match the oracle's
// sum of its rounded U_hat to ~1e-13. Roundings that repeat a pattern are replicated
// exactly: s*x (a fixed s times 8-bit bf16 mantissas) and, on the floor, the division
// by the constant D = sqrt(eps) (Markstein's correctly rounded division with the
// correctly rounded reciprocal). Above the floor the oracle's three roundings (of R_i c'_j,
// the square root and the quotient) vary freely from element to element, so U_hat is
// taken unrounded in double, and the sum of U_hat^4 over those elements gives the
// spread of the difference. The clip stage decides k from this; when the bound leaves
// k's rounding open, an exact pass (p2_exact) recomputes the tensor's sum.
// --------------------------------------------------------------------------------------------
struct SumPair {
  double s, q4;
};

__device__ __forceinline__ SumPair p2_factored(const DevTensor &t, const Tile &tl, const StepConsts &k, float q) {
  const WaveMap wm(t, tl);
  const int64_t m = t.m, ld = t.ld, col = wm.col;
  const bool mom = t.momentum != 0;
  const float s = mom ? k.s_m : k.s_0;
  const float deps = sqrtf(k.eps);                    // the oracle's D on the floor
  const float reps = (float)(1.0 / (double)deps);     // correctly rounded 1/D
  SumPair acc = {0.0, 0.0};
  if (col >= m) return acc;
  float cp[8];    // c'_j = C_j / q, rounded as the oracle
  double bd[8];   // 1/sqrt(c'_j)
#pragma unroll
  for (int e = 0; e < 8; e++) {
    cp[e] = (col + e < m) ? ldg(t.C + col + e) / q : 0.f;
    bd[e] = 1.0 / sqrt((double)cp[e]);
  }
  auto elem = [&](float x, float Ri, double ai, int e, SumPair &a) {
    const float ax = __fmul_rn(s, x);
    const bool floored = __fmul_rn(Ri, cp[e]) < k.eps;
    const float q0 = ax * reps;
    const float uf = fmaf(fmaf(-q0, deps, ax), reps, q0);   // RN(ax / deps)
    const double ud = (double)ax * (ai * bd[e]);
    const double u = floored ? (double)uf : ud;
    a.s = fma(u, u, a.s);
    const double u2 = floored ? 0.0 : ud * ud;
    a.q4 = fma(u2, u2, a.q4);
  };
  if (t.vec) {
    for (int64_t lr = wm.wr; lr < tl.nr; lr += 2 * wm.rpi) {
      const bool two = lr + wm.rpi < tl.nr;
      const int64_t i = tl.row(lr), i2 = two ? tl.row(lr + wm.rpi) : i;
      const uint4 ga = ldg(reinterpret_cast<const uint4 *>(t.g + i * ld + col));
      const uint4 gb = ldg(reinterpret_cast<const uint4 *>(t.g + i2 * ld + col));
      float ma[8], mb[8];
      if (mom) {
        load_m8(t.M + i * m + col, ma);
        load_m8(t.M + i2 * m + col, mb);
      }
      const float Ra = ldg(t.R + i), Rb = ldg(t.R + i2);
      const double aa = ldg(t.ainv + i), ab = ldg(t.ainv + i2);
      float xa[8], xb[8];
      unpack8(ga, xa);
      unpack8(gb, xb);
      if (mom) {
#pragma unroll
        for (int e = 0; e < 8; e++) {
          xa[e] = fmaf(k.a1, xa[e], __fmul_rn(k.b1, ma[e]));
          xb[e] = fmaf(k.a1, xb[e], __fmul_rn(k.b1, mb[e]));
        }
      }
      SumPair sa = {0.0, 0.0}, sb = {0.0, 0.0};
#pragma unroll
      for (int e = 0; e < 8; e++) {
        elem(xa[e], Ra, aa, e, sa);
        elem(xb[e], Rb, ab, e, sb);
      }
      acc.s += sa.s;
      acc.q4 += sa.q4;
      if (two) {
        acc.s += sb.s;
        acc.q4 += sb.q4;
      }
    }
  } else {
    for (int64_t lr = wm.wr; lr < tl.nr; lr += wm.rpi) {
      const int64_t i = tl.row(lr);
      const float Ri = ldg(t.R + i);
      const double ai = ldg(t.ainv + i);
#pragma unroll
      for (int e = 0; e < 8; e++) {
        if (col + e >= m) continue;
        float x = bf_one(ldg(t.g + i * ld + col + e));
        if (mom) x = fmaf(k.a1, x, __fmul_rn(k.b1, ldg(t.M + i * m + col + e)));
        elem(x, Ri, ai, e, acc);
      }
    }
  }
  return acc;
}

// The oracle's own float sequence for U_hat of a factored tensor, summed in double:
// used when the approximate sum leaves the clip factor's rounding undecided.
__device__ __forceinline__ double p2_factored_exact(const DevTensor &t, const Tile &tl, const StepConsts &k,
                                                    float q) {
  const WaveMap wm(t, tl);
  const int64_t m = t.m, ld = t.ld, col = wm.col;
  const bool mom = t.momentum != 0;
  const float s = mom ? k.s_m : k.s_0;
  double acc = 0.0;
  if (col >= m) return 0.0;
  float cp[8];
#pragma unroll
  for (int e = 0; e < 8; e++) cp[e] = (col + e < m) ? ldg(t.C + col + e) / q : 0.f;
  for (int64_t lr = wm.wr; lr < tl.nr; lr += wm.rpi) {
    const int64_t i = tl.row(lr);
    const float Ri = ldg(t.R + i);
#pragma unroll
    for (int e = 0; e < 8; e++) {
      if (col + e >= m) continue;
      float x = bf_one(ldg(t.g + i * ld + col + e));
      if (mom) x = fmaf(k.a1, x, __fmul_rn(k.b1, ldg(t.M + i * m + col + e)));
      const float u = __fmul_rn(s, x) / sqrtf(max_nan(__fmul_rn(Ri, cp[e]), k.eps));
      acc = fma((double)u, (double)u, acc);
    }
  }
  return acc;
}

__device__ __forceinline__ double p2_exact(const DevTensor &t, const Tile &tl, const StepConsts &k) {
  // exact second moment (router tier, vectors): the oracle's operation order exactly
  const WaveMap wm(t, tl);
  const int64_t m = t.m, ld = t.ld, col = wm.col;
  const bool mom = t.momentum != 0;
  double acc = 0.0;
  for (int64_t lr = wm.wr; lr < tl.nr; lr += wm.rpi) {
    const int64_t i = tl.row(lr);
#pragma unroll
    for (int e = 0; e < 8; e++) {
      if (col + e >= m) continue;
      const int64_t sidx = i * m + col + e;
      const float g = bf_one(ldg(t.g + i * ld + col + e));
      const float vn = fmaf(k.a2, __fmul_rn(g, g), __fmul_rn(k.b2, ldg(t.V + sidx)));
      const float dd = sqrtf(max_nan(vn, k.eps));
      const float num = mom ? __fmul_rn(k.s_m, fmaf(k.a1, g, __fmul_rn(k.b1, ldg(t.M + sidx)))) : __fmul_rn(k.s_0, g);
      const float u = num / dd;
      acc += (double)u * (double)u;
    }
  }
  return acc;
}

__global__ __launch_bounds__(kThreads) void p2_kernel(const DevTensor *__restrict__ TT,
                                                      const Item *__restrict__ items, StepConsts k) {
  __shared__ double sh[kThreads];
  const Item it = items[blockIdx.x];
  const DevTensor &t = TT[it.tensor];
  const Tile tl = tile_of(t, it.tile);
  SumPair acc;
  if (t.kind == kFactored) {
    const float q = mean_r_clamped(t, k.eps, sh);
    acc = p2_factored(t, tl, k, q);
  } else {
    acc.s = p2_exact(t, tl, k);   // already the oracle's own U_hat
    acc.q4 = 0.0;
  }
  const double s = block_sum(acc.s, sh);
  const double q4 = block_sum(acc.q4, sh);
  if (threadIdx.x == 0) {
    stg(t.ssum + it.tile, s);
    stg(t.qsum + it.tile, q4);
  }
}

// exact re-run of p2 for the tensors the clip stage left undecided (others exit at once)
__global__ __launch_bounds__(kThreads) void p2_exact_kernel(const DevTensor *__restrict__ TT,
                                                            const Item *__restrict__ items, StepConsts k) {
  __shared__ double sh[kThreads];
  const Item it = items[blockIdx.x];
  const DevTensor &t = TT[it.tensor];
  if (t.kind != kFactored || ldg(&t.sc->ambiguous) == 0) return;
  const Tile tl = tile_of(t, it.tile);
  const float q = mean_r_clamped(t, k.eps, sh);
  const double s = block_sum(p2_factored_exact(t, tl, k, q), sh);
  if (threadIdx.x == 0) stg(t.ssum + it.tile, s);
}

// --------------------------------------------------------------------------------------------
// clip stage, one work-group per tensor: k = 1 / max(1, RMS(U_hat) / d) (Sec. 3, Alg. 1),
// NaN-propagating and rounded once to float as the oracle rounds it. With exact == 0 it
// also records q = max(mean R, eps) and flags the tensor when the approximate sum's
// spread (20 standard deviations, from the sum of U_hat^4) reaches a rounding boundary
// of k or the clipping threshold; with exact == 1 it recomputes k of flagged tensors
// from the exact sums.
// --------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void clip_kernel(const DevTensor *__restrict__ TT,
                                                        const Item *__restrict__ items, StepConsts k, int exact) {
  __shared__ double sh[kThreads];
  const Item it = items[blockIdx.x];
  const DevTensor &t = TT[it.tensor];
  if (exact && ldg(&t.sc->ambiguous) == 0) return;
  const int64_t ntiles = (int64_t)t.ntr * t.ntc;
  const double S = wg_sum(t.ssum, ntiles, sh);
  const double Q4 = exact ? 0.0 : wg_sum(t.qsum, ntiles, sh);
  const float q = (!exact && t.kind == kFactored) ? mean_r_clamped(t, k.eps, sh) : 0.f;
  if (threadIdx.x != 0) return;
  const double r = sqrt(S / (double)(t.n * t.m)) / (double)k.d;
  const double den = (r != r) ? r : (r < 1.0 ? 1.0 : r);
  const double kd = 1.0 / den;
  const float kf = (float)kd;
  if (exact) {
    stg(&t.sc->k, kf);
    stg(&t.sc->ambiguous, 2);
    return;
  }
  bool amb = (k.flags & SKEW_FLAG_EXACT_CLIP) != 0 && t.kind == kFactored;
  if (S > 0.0 && r == r && r < 1e300) {
    const double spread = 20.0 * 0x1p-23 * sqrt(Q4) / S + 1e-14;   // relative, on S
    if (fabs(r - 1.0) <= spread) amb = true;                         // at the clipping threshold
    if (r > 1.0) {
      const double up = (double)nextafterf(kf, 3.0e38f), dn = (double)nextafterf(kf, 0.f);
      const double mid_hi = 0.5 * ((double)kf + up), mid_lo = 0.5 * ((double)kf + dn);
      const double tol = 0.5 * spread * kd;
      if (fabs(kd - mid_hi) <= tol || fabs(kd - mid_lo) <= tol) amb = true;
    }
  }
  stg(&t.sc->k, kf);
  stg(&t.sc->q, q);
  stg(&t.sc->ambiguous, amb ? 1 : 0);
}

// The oracle's float sequence for one factored element (Alg. 1 with the eps clamps):
// D = sqrt(max(R_i * c'_j, eps)), U = ((s * x) / D) * k, y = (w - lr U) + xi.
__device__ __forceinline__ float exact_factored_y(float x, float w, float Ri, float cpj, float s, float kc,
                                                  float eps, float lr, float dith) {
  const float vh = __fmul_rn(Ri, cpj);
  const float dd = sqrtf(max_nan(vh, eps));
  const float U = __fmul_rn(__fmul_rn(s, x) / dd, kc);
  return fmaf(dith, fabsf(w), fmaf(-lr, U, w));
}

// True when y may round differently from the oracle's value: the fast update x*F differs
// from the oracle's lr*U by < 2^-19 relative, and each of x and y carries one rounding.
__device__ __forceinline__ bool near_boundary(float y, float xF, float w) {
  const float mid = __uint_as_float((__float_as_uint(y) & 0xFFFF0000u) | 0x8000u);
  const float bound = fmaf(fabsf(xF), 0x1p-18f + 0x1p-21f, fabsf(w) * 0x1p-21f);
  return fabsf(y - mid) <= bound;
}

struct P3Scalars {
  float q, s, kc, cap3, eps, lr;
  double lsk;
};

// one row segment of 8 elements (vector path): momentum, update, dither, bf16 store.
// The fast path forms 1/D from per-row and per-column factors; the few elements whose
// result might round to the other bf16 neighbour take the oracle's exact sequence.
__device__ __forceinline__ void p3_row8(const DevTensor &t, const StepConsts &k, const P3Scalars &c,
                                        const Dither &dz, int64_t i, int64_t col, const float *bf, uint4 gw,
                                        uint4 ww, const float *mv) {
  const bool mom = t.momentum != 0;
  float x[8], w[8];
  unpack8(gw, x);
  unpack8(ww, w);
  if (mom) {
#pragma unroll
    for (int e = 0; e < 8; e++) x[e] = fmaf(k.a1, x[e], __fmul_rn(k.b1, mv[e]));
    store_m8(t.M + i * t.m + col, x);
  }
  const float alpha = (float)(c.lsk * ldg(t.ainv + i));
  const uint64_t p0 = ((uint64_t)i * (uint64_t)t.m + (uint64_t)col) >> 1;   // m and col are even here
  float y[8], dith[8];
  bool any = false;
#pragma unroll
  for (int e2 = 0; e2 < 4; e2++) {
    const uint32_t h = dz.pair(p0 + e2);
    dith[2 * e2] = dither_lo(h);
    dith[2 * e2 + 1] = dither_hi(h);
  }
#pragma unroll
  for (int e = 0; e < 8; e++) {
    const float F = fminf(alpha * bf[e], c.cap3);
    y[e] = fmaf(dith[e], fabsf(w[e]), fmaf(-x[e], F, w[e]));
    any |= near_boundary(y[e], x[e] * F, w[e]);
  }
  if (any) {
    const float Ri = ldg(t.R + i);
#pragma unroll
    for (int e = 0; e < 8; e++) {
      const float F = fminf(alpha * bf[e], c.cap3);
      if (near_boundary(y[e], x[e] * F, w[e]))
        y[e] = exact_factored_y(x[e], w[e], Ri, ldg(t.C + col + e) / c.q, c.s, c.kc, c.eps, c.lr, dith[e]);
    }
  }
  stg(reinterpret_cast<uint4 *>(t.w + i * t.ld + col),
      make_uint4(pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3]), pack_bf16x2(y[4], y[5]),
                 pack_bf16x2(y[6], y[7])));
}

__device__ __forceinline__ void p3_factored(const DevTensor &t, const Tile &tl, const StepConsts &k, float kc,
                                            float q, const Dither &dz) {
  const WaveMap wm(t, tl);
  const int64_t m = t.m, ld = t.ld, col = wm.col;
  const bool mom = t.momentum != 0;
  if (col >= m) return;
  P3Scalars c;
  c.q = q;
  c.s = mom ? k.s_m : k.s_0;
  c.kc = kc;
  c.eps = k.eps;
  c.lr = k.lr;
  c.lsk = (double)k.lr * (double)c.s * (double)kc;   // lr * s * k
  c.cap3 = (float)(c.lsk / (double)sqrtf(k.eps));
  if (t.vec) {
    float bf[8];
#pragma unroll
    for (int e = 0; e < 8; e++) bf[e] = (float)col_factor(t, col + e, c.q);
    for (int64_t lr = wm.wr; lr < tl.nr; lr += 2 * wm.rpi) {
      const bool two = lr + wm.rpi < tl.nr;
      const int64_t i = tl.row(lr), i2 = two ? tl.row(lr + wm.rpi) : i;
      const uint4 ga = ldg(reinterpret_cast<const uint4 *>(t.g + i * ld + col));
      const uint4 wa = ldg(reinterpret_cast<const uint4 *>(t.w + i * ld + col));
      const uint4 gb = ldg(reinterpret_cast<const uint4 *>(t.g + i2 * ld + col));
      const uint4 wb = ldg(reinterpret_cast<const uint4 *>(t.w + i2 * ld + col));
      float ma[8], mb[8];
      if (mom) {
        load_m8(t.M + i * m + col, ma);
        load_m8(t.M + i2 * m + col, mb);
      }
      p3_row8(t, k, c, dz, i, col, bf, ga, wa, ma);
      if (two) p3_row8(t, k, c, dz, i2, col, bf, gb, wb, mb);
    }
  } else {
    for (int64_t lr = wm.wr; lr < tl.nr; lr += wm.rpi) {
    const int64_t i = tl.row(lr);
      const float alpha = (float)(c.lsk * ldg(t.ainv + i));
      const uint64_t rowidx = (uint64_t)i * (uint64_t)m;
#pragma unroll
      for (int e = 0; e < 8; e++) {
        if (col + e >= m) continue;
        float x = bf_one(ldg(t.g + i * ld + col + e));
        const float w = bf_one(ldg(t.w + i * ld + col + e));
        if (mom) {
          x = fmaf(k.a1, x, __fmul_rn(k.b1, ldg(t.M + i * m + col + e)));
          stg(t.M + i * m + col + e, x);
        }
        const uint64_t idx = rowidx + (uint64_t)(col + e);
        const float dith = dither_of(dz.pair(idx >> 1), idx);
        const float F = fminf(alpha * (float)col_factor(t, col + e, c.q), c.cap3);
        float y = fmaf(dith, fabsf(w), fmaf(-x, F, w));
        if (near_boundary(y, x * F, w))
          y = exact_factored_y(x, w, ldg(t.R + i), ldg(t.C + col + e) / c.q, c.s, kc, k.eps, k.lr, dith);
        stg(t.w + i * ld + col + e, to_bf16(y));
      }
    }
  }
}

__device__ __forceinline__ void p3_exact(const DevTensor &t, const Tile &tl, const StepConsts &k, float kc,
                                         const Dither &dz) {
  // exact second moment: the oracle's operation order exactly
  const WaveMap wm(t, tl);
  const int64_t m = t.m, ld = t.ld, col = wm.col;
  const bool mom = t.momentum != 0;
  for (int64_t lr = wm.wr; lr < tl.nr; lr += wm.rpi) {
    const int64_t i = tl.row(lr);
#pragma unroll
    for (int e = 0; e < 8; e++) {
      if (col + e >= m) continue;
      const int64_t sidx = i * m + col + e;
      const float g = bf_one(ldg(t.g + i * ld + col + e));
      const float w = bf_one(ldg(t.w + i * ld + col + e));
      const float vn = fmaf(k.a2, __fmul_rn(g, g), __fmul_rn(k.b2, ldg(t.V + sidx)));
      stg(t.V + sidx, vn);
      const float dd = sqrtf(max_nan(vn, k.eps));
      float num;
      if (mom) {
        const float mn = fmaf(k.a1, g, __fmul_rn(k.b1, ldg(t.M + sidx)));
        stg(t.M + sidx, mn);
        num = __fmul_rn(k.s_m, mn);
      } else {
        num = __fmul_rn(k.s_0, g);
      }
      const float U = __fmul_rn(num / dd, kc);
      const float x = fmaf(-k.lr, U, w);
      const uint64_t idx = (uint64_t)sidx;
      const float y = fmaf(dither_of(dz.pair(idx >> 1), idx), fabsf(w), x);
      stg(t.w + i * ld + col + e, to_bf16(y));
    }
  }
}

// --------------------------------------------------------------------------------------------
// p3: clip factor, state update, weight update and dithered bf16 write-back (Alg. 1)
// --------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void p3_kernel(const DevTensor *__restrict__ TT,
                                                      const Item *__restrict__ items, StepConsts k) {
  const Item it = items[blockIdx.x];
  const DevTensor &t = TT[it.tensor];
  const Tile tl = tile_of(t, it.tile);
  const float kc = ldg(&t.sc->k);
  const Dither dz(k.seed, k.step, t.tensor_id);
  if (t.kind == kFactored)
    p3_factored(t, tl, k, kc, ldg(&t.sc->q), dz);
  else
    p3_exact(t, tl, k, kc, dz);
}

}  // namespace

int launch_p1(const DevTensor *T, const Item *items, int64_t count, void *stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(p1_kernel, dim3((uint32_t)count), dim3(kThreads), 0, (hipStream_t)stream, T, items);
  return (int)hipGetLastError();
}
int launch_fold(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, void *stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(fold_kernel, dim3((uint32_t)count), dim3(kThreads), 0, (hipStream_t)stream, T, items, k);
  return (int)hipGetLastError();
}
int launch_p2(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, void *stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(p2_kernel, dim3((uint32_t)count), dim3(kThreads), 0, (hipStream_t)stream, T, items, k);
  return (int)hipGetLastError();
}
int launch_clip(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, int exact, void *stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(clip_kernel, dim3((uint32_t)count), dim3(kThreads), 0, (hipStream_t)stream, T, items, k, exact);
  return (int)hipGetLastError();
}
int launch_p2_exact(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, void *stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(p2_exact_kernel, dim3((uint32_t)count), dim3(kThreads), 0, (hipStream_t)stream, T, items, k);
  return (int)hipGetLastError();
}
int launch_p3(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, void *stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(p3_kernel, dim3((uint32_t)count), dim3(kThreads), 0, (hipStream_t)stream, T, items, k);
  return (int)hipGetLastError();
}

}  // namespace skew
