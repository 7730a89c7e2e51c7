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

struct Tile {
  int64_t r0, r1, c0;
  int band, strip;
};
__device__ __forceinline__ Tile tile_of(const DevTensor &t, int tile) {
  Tile g;
  g.band = tile / t.ntc;
  g.strip = tile - g.band * t.ntc;
  g.r0 = (int64_t)g.band * t.tr;
  g.r1 = min(t.n, g.r0 + t.tr);
  g.c0 = (int64_t)g.strip * kChunk * t.cw;
  return g;
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

__global__ __launch_bounds__(kThreads) void p1_kernel(const DevTensor *__restrict__ TT,
                                                      const Item *__restrict__ items) {
  __shared__ double sh[2][kChunk * kMaxCw];
  const Item it = items[blockIdx.x];
  const DevTensor &t = TT[it.tensor];
  const Tile tl = tile_of(t, it.tile);
  const int64_t n = t.n, m = t.m, ld = t.ld;
  const int cw = t.cw;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const uint16_t *__restrict__ G = t.g;

  double acc[kMaxCw][8];
#pragma unroll
  for (int q = 0; q < kMaxCw; q++)
#pragma unroll
    for (int e = 0; e < 8; e++) acc[q][e] = 0.0;

  for (int64_t i = tl.r0 + wave; i < tl.r1; i += kWaves) {
    const uint16_t *row = G + i * ld;
    double rs = 0.0;
#pragma unroll
    for (int q = 0; q < kMaxCw; q++) {
      if (q < cw) {
        const int64_t col = tl.c0 + q * kChunk + lane * 8;
        float g[8];
        if (t.vec) {
          if (col < m) {
            unpack8(*reinterpret_cast<const uint4 *>(row + col), g);
          } else {
#pragma unroll
            for (int e = 0; e < 8; e++) g[e] = 0.f;
          }
        } else {
#pragma unroll
          for (int e = 0; e < 8; e++) g[e] = (col + e < m) ? bf_one(row[col + e]) : 0.f;
        }
#pragma unroll
        for (int e = 0; e < 8; e++) {
          const double gd = (double)g[e];
          rs = fma(gd, gd, rs);
          acc[q][e] = fma(gd, gd, acc[q][e]);
        }
      }
    }
    rs = wave_sum_d(rs);
    if (lane == 0) t.rowpart[(int64_t)tl.strip * n + i] = rs;
  }
  // column partials of the four waves: (w0 + w2) + (w1 + w3)
  if (wave >= 2) {
#pragma unroll
    for (int q = 0; q < kMaxCw; q++)
      if (q < cw)
#pragma unroll
        for (int e = 0; e < 8; e++) sh[wave - 2][q * kChunk + lane * 8 + e] = acc[q][e];
  }
  __syncthreads();
  if (wave < 2) {
#pragma unroll
    for (int q = 0; q < kMaxCw; q++)
      if (q < cw)
#pragma unroll
        for (int e = 0; e < 8; e++) acc[q][e] += sh[wave][q * kChunk + lane * 8 + e];
  }
  __syncthreads();
  if (wave == 1) {
#pragma unroll
    for (int q = 0; q < kMaxCw; q++)
      if (q < cw)
#pragma unroll
        for (int e = 0; e < 8; e++) sh[0][q * kChunk + lane * 8 + e] = acc[q][e];
  }
  __syncthreads();
  if (wave == 0) {
#pragma unroll
    for (int q = 0; q < kMaxCw; q++) {
      if (q >= cw) continue;
#pragma unroll
      for (int e = 0; e < 8; e++) {
        const int64_t col = tl.c0 + q * kChunk + lane * 8 + e;
        if (col < m) t.colpart[(int64_t)tl.band * m + col] = acc[q][e] + sh[0][q * kChunk + lane * 8 + e];
      }
    }
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
      for (int q = 0; q < t.ntc; q++) s += t.rowpart[(int64_t)q * t.n + i];
      const float ri = (float)(s / (double)t.m);
      const float R = fmaf(k.a2, ri, __fmul_rn(k.b2, t.R[i]));
      t.R[i] = R;
      t.ainv[i] = 1.0 / sqrt((double)R);
      rn = (double)R;
    }
    const double tot = block_sum(rn, sh);
    if (threadIdx.x == 0) t.rsum[it.tile] = tot;
  } else {
    const int64_t j = (int64_t)(it.tile - t.nfr) * kFold + threadIdx.x;
    if (j < t.m) {
      double s = 0.0;
      for (int b = 0; b < t.ntr; b++) s += t.colpart[(int64_t)b * t.m + j];
      const float cj = (float)(s / (double)t.n);
      t.C[j] = fmaf(k.a2, cj, __fmul_rn(k.b2, t.C[j]));
    }
  }
}

// Column factors of the rank-one reconstruction for one tile: q = max(mean R, eps) and
// c'_j = C_j / q exactly as the oracle rounds them, and b_j = 1/sqrt(c'_j) in double,
// so that 1/D_ij = min(b_j / sqrt(R_i), 1/sqrt(eps)) (Eq. 1 reconstruction, Alg. 1 clamps).
__device__ __forceinline__ float mean_r_clamped(const DevTensor &t, float eps) {
  double sr = 0.0;
  for (int c = 0; c < t.nfr; c++) sr += t.rsum[c];
  return max_nan((float)(sr / (double)t.n), eps);
}
__device__ __forceinline__ void column_factors(const DevTensor &t, const Tile &tl, float q, double (&bd)[kMaxCw][8]) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int qq = 0; qq < kMaxCw; qq++)
#pragma unroll
    for (int e = 0; e < 8; e++) {
      const int64_t col = tl.c0 + qq * kChunk + lane * 8 + e;
      bd[qq][e] = (qq < t.cw && col < t.m) ? 1.0 / sqrt((double)(t.C[col] / q)) : 0.0;
    }
}

// --------------------------------------------------------------------------------------------
// p2: per-tile sum of squares of the unclipped update U_hat (Alg. 1, before clipping), in
// double from the unrounded U_hat; it differs from the oracle's sum of rounded U_hat by
// about 1e-8 / sqrt(N) relative, so the clip factor rounds to the same float.
// --------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void p2_kernel(const DevTensor *__restrict__ TT,
                                                      const Item *__restrict__ items, StepConsts k) {
  __shared__ double sh[kThreads];
  const Item it = items[blockIdx.x];
  const DevTensor &t = TT[it.tensor];
  const Tile tl = tile_of(t, it.tile);
  const int64_t m = t.m, ld = t.ld;
  const int cw = t.cw;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const bool mom = t.momentum != 0;
  double acc = 0.0;

  if (t.kind == kFactored) {
    const float q = mean_r_clamped(t, k.eps);
    double bd[kMaxCw][8];
    column_factors(t, tl, q, bd);
    const double sd = (double)(mom ? k.s_m : k.s_0);
    const double capd = sd / (double)sqrtf(k.eps);   // s / D at the floor, with the oracle's D
    for (int64_t i = tl.r0 + wave; i < tl.r1; i += kWaves) {
      const double alpha = sd * t.ainv[i];
      const uint16_t *grow = t.g + i * ld;
      const float *mrow = mom ? t.M + i * m : nullptr;
#pragma unroll
      for (int q = 0; q < kMaxCw; q++) {
        if (q >= cw) continue;
        const int64_t col = tl.c0 + q * kChunk + lane * 8;
        if (t.vec) {
          if (col >= m) continue;
          float x[8];
          unpack8(*reinterpret_cast<const uint4 *>(grow + col), x);
          if (mom) {
            const float4 m0 = *reinterpret_cast<const float4 *>(mrow + col);
            const float4 m1 = *reinterpret_cast<const float4 *>(mrow + col + 4);
            const float mv[8] = {m0.x, m0.y, m0.z, m0.w, m1.x, m1.y, m1.z, m1.w};
#pragma unroll
            for (int e = 0; e < 8; e++) x[e] = fmaf(k.a1, x[e], __fmul_rn(k.b1, mv[e]));
          }
#pragma unroll
          for (int e = 0; e < 8; e++) {
            const double u = (double)x[e] * fmin(alpha * bd[q][e], capd);
            acc = fma(u, u, acc);
          }
        } else {
#pragma unroll
          for (int e = 0; e < 8; e++) {
            if (col + e >= m) continue;
            float x = bf_one(grow[col + e]);
            if (mom) x = fmaf(k.a1, x, __fmul_rn(k.b1, mrow[col + e]));
            const double u = (double)x * fmin(alpha * bd[q][e], capd);
            acc = fma(u, u, acc);
          }
        }
      }
    }
  } else {
    // exact second moment (router tier, vectors): the oracle's operation order exactly
    for (int64_t i = tl.r0 + wave; i < tl.r1; i += kWaves) {
      const uint16_t *grow = t.g + i * ld;
#pragma unroll
      for (int q = 0; q < kMaxCw; q++) {
        if (q >= cw) continue;
        const int64_t col = tl.c0 + q * kChunk + lane * 8;
#pragma unroll
        for (int e = 0; e < 8; e++) {
          if (col + e >= m) continue;
          const int64_t sidx = i * m + col + e;
          const float g = bf_one(grow[col + e]);
          const float vn = fmaf(k.a2, __fmul_rn(g, g), __fmul_rn(k.b2, t.V[sidx]));
          const float dd = sqrtf(max_nan(vn, k.eps));
          const float num = mom ? __fmul_rn(k.s_m, fmaf(k.a1, g, __fmul_rn(k.b1, t.M[sidx]))) : __fmul_rn(k.s_0, g);
          const float u = num / dd;
          acc += (double)u * (double)u;
        }
      }
    }
  }
  const double tot = block_sum(acc, sh);
  if (threadIdx.x == 0) t.ssum[it.tile] = tot;
}

// The oracle's float sequence for one factored element (Alg. 1 with the eps clamps):
// D = sqrt(max(R_i * c'_j, eps)), U = ((s * x) / D) * k, y = (w - lr U) + xi.
__device__ __attribute__((noinline)) float exact_factored_y(float x, float w, float Ri, float cpj, float s, float kc,
                                                            float eps, float lr, float dith) {
  const float vh = __fmul_rn(Ri, cpj);
  const float dd = sqrtf(max_nan(vh, eps));
  const float U = __fmul_rn(__fmul_rn(s, x) / dd, kc);
  return fmaf(dith, fabsf(w), fmaf(-lr, U, w));
}

// True when y may round differently from the oracle's value: the fast update g*F differs
// from the oracle's lr*U by < 2^-19 relative, and each of x and y carries one rounding.
__device__ __forceinline__ bool near_boundary(float y, float gF, float w) {
  const float mid = __uint_as_float((__float_as_uint(y) & 0xFFFF0000u) | 0x8000u);
  const float bound = fmaf(fabsf(gF), 0x1p-18f + 0x1p-21f, fabsf(w) * 0x1p-21f);
  return fabsf(y - mid) <= bound;
}

// --------------------------------------------------------------------------------------------
// p3: clip factor, state update, weight update and dithered bf16 write-back (Alg. 1)
// --------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void p3_kernel(const DevTensor *__restrict__ TT,
                                                      const Item *__restrict__ items, StepConsts k) {
  const Item it = items[blockIdx.x];
  const DevTensor &t = TT[it.tensor];
  const Tile tl = tile_of(t, it.tile);
  const int64_t m = t.m, ld = t.ld;
  const int cw = t.cw;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const bool mom = t.momentum != 0;

  // clip factor k = 1 / max(1, RMS(U_hat) / d), NaN-propagating, rounded once as the oracle
  double S = 0.0;
  const int ntiles = t.ntr * t.ntc;
  for (int c = 0; c < ntiles; c++) S += t.ssum[c];
  const double ratio = sqrt(S / (double)(t.n * m)) / (double)k.d;
  const double den = (ratio != ratio) ? ratio : (ratio < 1.0 ? 1.0 : ratio);
  const float kc = (float)(1.0 / den);
  const Dither dz(k.seed, k.step, t.tensor_id);

  if (t.kind == kFactored) {
    const float q = mean_r_clamped(t, k.eps);
    float bf[kMaxCw][8];
    {
      double bd[kMaxCw][8];
      column_factors(t, tl, q, bd);
#pragma unroll
      for (int qq = 0; qq < kMaxCw; qq++)
#pragma unroll
        for (int e = 0; e < 8; e++) bf[qq][e] = (float)bd[qq][e];
    }
    const float s = mom ? k.s_m : k.s_0;
    const double lsk = (double)k.lr * (double)s * (double)kc;   // lr * s * k
    const float cap3 = (float)(lsk / (double)sqrtf(k.eps));
    for (int64_t i = tl.r0 + wave; i < tl.r1; i += kWaves) {
      const float alpha = (float)(lsk * t.ainv[i]);
      const float Ri = t.R[i];
      const uint16_t *grow = t.g + i * ld;
      uint16_t *wrow = t.w + i * ld;
      float *mrow = mom ? t.M + i * m : nullptr;
      const uint64_t rowidx = (uint64_t)i * (uint64_t)m;
#pragma unroll
      for (int qc = 0; qc < kMaxCw; qc++) {
        if (qc >= cw) continue;
        const int64_t col = tl.c0 + qc * kChunk + lane * 8;
        if (t.vec) {
          if (col >= m) continue;
          float x[8], w[8];
          unpack8(*reinterpret_cast<const uint4 *>(grow + col), x);
          unpack8(*reinterpret_cast<const uint4 *>(wrow + col), w);
          if (mom) {
            const float4 m0 = *reinterpret_cast<const float4 *>(mrow + col);
            const float4 m1 = *reinterpret_cast<const float4 *>(mrow + col + 4);
            const float mv[8] = {m0.x, m0.y, m0.z, m0.w, m1.x, m1.y, m1.z, m1.w};
#pragma unroll
            for (int e = 0; e < 8; e++) x[e] = fmaf(k.a1, x[e], __fmul_rn(k.b1, mv[e]));
            *reinterpret_cast<float4 *>(mrow + col) = make_float4(x[0], x[1], x[2], x[3]);
            *reinterpret_cast<float4 *>(mrow + col + 4) = make_float4(x[4], x[5], x[6], x[7]);
          }
          const uint64_t p0 = (rowidx + (uint64_t)col) >> 1;   // m and col are even here
          uint32_t out[4];
#pragma unroll
          for (int e2 = 0; e2 < 4; e2++) {
            const uint32_t h = dz.pair(p0 + e2);
            float y[2];
#pragma unroll
            for (int h2 = 0; h2 < 2; h2++) {
              const int e = 2 * e2 + h2;
              const float dith = h2 ? dither_hi(h) : dither_lo(h);
              const float F = fminf(alpha * bf[qc][e], cap3);
              const float yf = fmaf(dith, fabsf(w[e]), fmaf(-x[e], F, w[e]));
              y[h2] = yf;
              if (near_boundary(yf, x[e] * F, w[e]))
                y[h2] = exact_factored_y(x[e], w[e], Ri, t.C[col + e] / q, s, kc, k.eps, k.lr, dith);
            }
            out[e2] = pack_bf16x2(y[0], y[1]);
          }
          *reinterpret_cast<uint4 *>(wrow + col) = make_uint4(out[0], out[1], out[2], out[3]);
        } else {
#pragma unroll
          for (int e = 0; e < 8; e++) {
            if (col + e >= m) continue;
            float x = bf_one(grow[col + e]);
            const float w = bf_one(wrow[col + e]);
            if (mom) {
              x = fmaf(k.a1, x, __fmul_rn(k.b1, mrow[col + e]));
              mrow[col + e] = x;
            }
            const uint64_t idx = rowidx + (uint64_t)(col + e);
            const float dith = dither_of(dz.pair(idx >> 1), idx);
            const float F = fminf(alpha * bf[qc][e], cap3);
            float y = fmaf(dith, fabsf(w), fmaf(-x, F, w));
            if (near_boundary(y, x * F, w)) y = exact_factored_y(x, w, Ri, t.C[col + e] / q, s, kc, k.eps, k.lr, dith);
            wrow[col + e] = to_bf16(y);
          }
        }
      }
    }
  } else {
    // exact second moment: the oracle's operation order exactly
    for (int64_t i = tl.r0 + wave; i < tl.r1; i += kWaves) {
      const uint16_t *grow = t.g + i * ld;
      uint16_t *wrow = t.w + i * ld;
#pragma unroll
      for (int q = 0; q < kMaxCw; q++) {
        if (q >= cw) continue;
        const int64_t col = tl.c0 + q * kChunk + lane * 8;
#pragma unroll
        for (int e = 0; e < 8; e++) {
          if (col + e >= m) continue;
          const int64_t sidx = i * m + col + e;
          const float g = bf_one(grow[col + e]);
          const float w = bf_one(wrow[col + e]);
          const float vn = fmaf(k.a2, __fmul_rn(g, g), __fmul_rn(k.b2, t.V[sidx]));
          t.V[sidx] = vn;
          const float dd = sqrtf(max_nan(vn, k.eps));
          float num;
          if (mom) {
            const float mn = fmaf(k.a1, g, __fmul_rn(k.b1, t.M[sidx]));
            t.M[sidx] = mn;
            num = __fmul_rn(k.s_m, mn);
          } else {
            num = __fmul_rn(k.s_0, g);
          }
          const float U = __fmul_rn(num / dd, kc);
          const float x = fmaf(-k.lr, U, w);
          const uint64_t idx = (uint64_t)sidx;
          const float y = fmaf(dither_of(dz.pair(idx >> 1), idx), fabsf(w), x);
          wrow[col + e] = to_bf16(y);
        }
      }
    }
  }
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
int launch_p3(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, void *stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(p3_kernel, dim3((uint32_t)count), dim3(kThreads), 0, (hipStream_t)stream, T, items, k);
  return (int)hipGetLastError();
}

}  // namespace skew
