// skew_kernels.hip -- gfx950 kernels of one SkewAdam step (Sec. 3, Eq. 1, Alg. 1).
//
// A step is a short sequence of stream-ordered launches over device-resident work-item
// tables; each launch covers every tensor of the table (e.g. all experts of a layer):
//   p1z   factored matrices up to 16384 columns (row-band pass): R_i, partial column sums
//         of g^2 and of (s x)^2 / R_i, the floored sum of U_hat^2 and bounds, in one read of G
//   p1    wider factored matrices: per tile, partial row and column sums of g^2 (Eq. 1)
//   fold  factored tensors: C (and for wide ones R) EMA (Eq. 1), 1/sqrt(R_i), c'_j and
//         the row-band tensors' sum of U_hat^2 above the floor
//   p2    exact-second-moment tensors and wide factored ones: per tile, sum of squares of
//         the unclipped update (Alg. 1)
//   clip  per tensor: the clip factor k, and whether its rounding needs the exact pass
//         (the slices of stacked tensors first, one wave each, in a launch of their own)
//   p2x   re-runs of the sum for the tensors the clip stage left undecided (the exact floor
//         split, then the oracle's float sequence); clip again
//   p3    every tensor: momentum / exact-v update, weight update, dithered bf16
//         write-back (Sec. 3 "Update clipping and low-precision updates")
// Reductions are deterministic (fixed-order partials; no float atomics), so two
// runs on the same inputs produce identical bits.
//
// Tile (p1, p2, p3): tr rows x (512*cw) columns. A work-group is 4 wave64; lane l covers 8
// consecutive columns (one 16-byte bf16 load) in each 512-column chunk.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <mutex>
#include <type_traits>

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
__device__ __forceinline__ void stg(float4 *p, float4 v) {
  const f32x4_t u = {v.x, v.y, v.z, v.w};
  stg(reinterpret_cast<f32x4_t *>(p), u);
}
// Non-temporal 16-byte loads and stores, for the bf16 gradient and weight rows that the update
// pass streams through once (a hint to the caches not to keep them). Together they took the
// 6.78B update pass from 8.07 to 7.65 ms; loads alone (8.23) or stores alone (8.12) did not,
// and on the fp32 momentum the hint costs time (the expert-momentum variant: 18.1 -> 19.2 ms).
template <class V>
__device__ __forceinline__ V ldg_nt(const V *p) {
  return __builtin_nontemporal_load((const __attribute__((address_space(1))) V *)p);
}
template <class V>
__device__ __forceinline__ void stg_nt(V *p, V v) {
  __builtin_nontemporal_store(v, (__attribute__((address_space(1))) V *)p);
}
__device__ __forceinline__ uint4 ldg_nt(const uint4 *p) {
  const u32x4_t v = ldg_nt(reinterpret_cast<const u32x4_t *>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void stg_nt(uint4 *p, uint4 v) {
  const u32x4_t u = {v.x, v.y, v.z, v.w};
  stg_nt(reinterpret_cast<u32x4_t *>(p), u);
}

__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xFFFF0000u); }
__device__ __forceinline__ float bf_one(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
// element idx of a weight or gradient array: bf16, or float32 for float32 masters
__device__ __forceinline__ float elem(const uint16_t *p, int64_t idx, bool fp32) {
  return fp32 ? ldg(reinterpret_cast<const float *>(p) + idx) : bf_one(ldg(p + idx));
}

// max(a, b) that returns `a` when it is NaN (b is a finite constant): NaN propagates.
__device__ __forceinline__ float max_nan(float a, float b) { return (a < b) ? b : a; }

__device__ __forceinline__ void unpack8(const uint4 &u, float *o) {
  o[0] = bf_lo(u.x); o[1] = bf_hi(u.x);
  o[2] = bf_lo(u.y); o[3] = bf_hi(u.y);
  o[4] = bf_lo(u.z); o[5] = bf_hi(u.z);
  o[6] = bf_lo(u.w); o[7] = bf_hi(u.w);
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
  // the hash input of pair p before the final mix: pair(p) = fmix32(pair_base(p))
  __device__ __forceinline__ uint32_t pair_base(uint64_t p) const {
    const uint32_t ph = (uint32_t)(p >> 32);
    const uint32_t inner = (ph == 0u) ? inner0 : fmix32(ph ^ khi);
    return (uint32_t)p ^ klo ^ inner;
  }
  __device__ __forceinline__ uint32_t pair(uint64_t p) const { return fmix32(pair_base(p)); }
};

// e * 2^-24 with e = 2*u16 + 1 - 2^16 = u16 * 2^-23 + (1 - 2^16) * 2^-24: a multiple of
// 2^-24 below 2^-8 in magnitude, so the fma is exact (u16 converts exactly)
__device__ __forceinline__ float dither_u16(uint32_t u) { return fmaf((float)u, 0x1p-23f, -65535.0f * 0x1p-24f); }
__device__ __forceinline__ float dither_lo(uint32_t h) { return dither_u16(h & 0xFFFFu); }
__device__ __forceinline__ float dither_hi(uint32_t h) { return dither_u16(h >> 16); }
__device__ __forceinline__ float dither_of(uint32_t h, uint64_t idx) { return (idx & 1u) ? dither_hi(h) : dither_lo(h); }

// The noise added before the cast is the product of two exact factors: e 2^-24 and |w|
// (ulp(w) taken as 2^-7 |w|, Sec. 3), or, in the exact-ulp mode, e 2^-24 and 2^7 times the
// bf16 ulp of w. That ulp is 2^(E - 134) for biased exponent E >= 1 and 2^-133 among the
// subnormals, so 2^7 ulp is the float whose exponent field is E clamped to [1, 254] (an
// infinite or NaN w keeps a finite factor; its update is infinite or NaN already)
__device__ __forceinline__ float bf16_ulp128(float w) {
  const uint32_t b = __float_as_uint(w) & 0x7F800000u;
  return __uint_as_float(min(max(b, 0x00800000u), 0x7F000000u));
}
__device__ __forceinline__ float dither_mul(float w, bool xu) { return xu ? bf16_ulp128(w) : fabsf(w); }

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

// Butterfly reductions over one wave64: every lane ends with the same value (each step
// adds two equal-order partials, and IEEE addition is commutative), so the result is
// deterministic.
__device__ __forceinline__ double wave_sum_d(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
  return x;
}
__device__ __forceinline__ double wave_max_d(double x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmax(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ __forceinline__ float wave_min_f(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fminf(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ __forceinline__ float wave_max_f(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}
__device__ __forceinline__ int wave_or(int x) { return __any(x != 0) ? 1 : 0; }

// Work-group reductions of NW waves through sh[NW] (every thread gets the result; the
// per-wave results are combined in wave order).
template <int NW>
__device__ __forceinline__ double wg_sum_w(double x, double *sh) {
  x = wave_sum_d(x);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = x;
  __syncthreads();
  double r = 0.0;
#pragma unroll
  for (int w = 0; w < NW; w++) r += sh[w];
  __syncthreads();
  return r;
}
template <int NW>
__device__ __forceinline__ double wg_max_w(double x, double *sh) {
  x = wave_max_d(x);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = x;
  __syncthreads();
  double r = sh[0];
#pragma unroll
  for (int w = 1; w < NW; w++) r = fmax(r, sh[w]);
  __syncthreads();
  return r;
}
template <int NW>
__device__ __forceinline__ float wg_min_wf(float x, double *sh) {
  x = wave_min_f(x);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = (double)x;
  __syncthreads();
  float r = (float)sh[0];
#pragma unroll
  for (int w = 1; w < NW; w++) r = fminf(r, (float)sh[w]);
  __syncthreads();
  return r;
}
template <int NW>
__device__ __forceinline__ float wg_max_wf(float x, double *sh) {
  x = wave_max_f(x);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = (double)x;
  __syncthreads();
  float r = (float)sh[0];
#pragma unroll
  for (int w = 1; w < NW; w++) r = fmaxf(r, (float)sh[w]);
  __syncthreads();
  return r;
}
template <int NW>
__device__ __forceinline__ int wg_or_w(int x, double *sh) {
  x = wave_or(x);
  if ((threadIdx.x & 63) == 0) sh[threadIdx.x >> 6] = (double)x;
  __syncthreads();
  int r = 0;
#pragma unroll
  for (int w = 0; w < NW; w++) r |= (sh[w] != 0.0) ? 1 : 0;
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
// Row-band pass: pass 1 of factored matrices whose staged rows fit (Eq. 1 and the update
// sum of Alg. 1 in one read of G).
//
// A work-group owns a band of whole rows, so R_i <- b2 R_i + a2 mean_j g_ij^2 is final as
// soon as row i is summed. With the row still at hand the work-group adds (s x_ij)^2 / R_i
// to a per-column sum z_j (x = g, or the new momentum on the backbone). Above the eps
// floor U_hat_ij^2 = (s x_ij)^2 / (R_i c'_j) up to the oracle's free roundings, so the
// tensor's sum of U_hat^2 is sum_j z_j / c'_j once the fold has c'_j = C_j / max(mean R,
// eps): no pass re-reads G for it. On the floor U_hat = RN(RN(s x) / sqrt(eps)) depends on
// x alone; its square is summed exactly as the oracle rounds it (Markstein's correctly
// rounded division). The clip stage takes whichever sum applies; the last step's
// regime decides which of the two this pass forms (a tensor that was clearly above the
// floor skips the floored sum, and the reverse).
//
// Roundings that repeat a pattern are replicated (RN(s x); the momentum fma), so the
// remaining difference from the oracle's sum is the free roundings of R_i c'_j, the
// square root and the quotient; the per-band maximum of (s x)^2 / R_i bounds their spread.
//
// Staging: blocks of zrpi * zrb whole rows (bf16 gradient, and fp32 momentum on the
// backbone). Aligned rows without momentum and with one or two chunks per wave (the normal
// step, and the gradient-norm mode's two passes) stage in registers: each wave loads its own
// pieces of the next block by buffer loads while it sums the current one. The other variants
// move a block into one of two LDS buffers while the other is being summed: with the direct
// global-to-LDS loads (16 bytes per lane) when rows are 16-byte aligned, through registers
// otherwise; no register holds their data in flight, so a 512-thread work-group with up to
// 256 VGPRs per wave keeps a whole block (up to 64 KiB) of loads outstanding.
//
// Layout: zcw 512-column chunks per row; a group of wpr = ceil(zcw / NSEG) waves shares a
// row, wave w of the group taking chunks w, w + wpr, ...; zrpi = 8 / wpr groups work on
// different rows. The column partials of the groups are added in group order through LDS.
// --------------------------------------------------------------------------------------------
__device__ __forceinline__ uint4 load_bf8(const uint16_t *base, int64_t ld, int64_t m, int64_t i, int64_t col) {
  const uint16_t *row = base + i * ld;
  uint32_t v[4];
#pragma unroll
  for (int e2 = 0; e2 < 4; e2++) {
    const uint32_t lo = (col + 2 * e2 < m) ? (uint32_t)ldg(row + col + 2 * e2) : 0u;
    const uint32_t hi = (col + 2 * e2 + 1 < m) ? (uint32_t)ldg(row + col + 2 * e2 + 1) : 0u;
    v[e2] = lo | (hi << 16);
  }
  return make_uint4(v[0], v[1], v[2], v[3]);
}

typedef __attribute__((address_space(3))) void lds_void_t;
typedef const __attribute__((address_space(1))) void gbl_void_t;
__device__ __forceinline__ void dma16(const void *g, void *lds) {
  __builtin_amdgcn_global_load_lds((gbl_void_t *)g, (lds_void_t *)lds, 16, 0, 0);
}
__device__ __forceinline__ void dma4(const void *g, void *lds) {
  __builtin_amdgcn_global_load_lds((gbl_void_t *)g, (lds_void_t *)lds, 4, 0, 0);
}
// s_waitcnt immediates (gfx9 encoding): vmcnt(0) and lgkmcnt(0); only lgkmcnt(0)
constexpr int kWaitVmLgkm0 = 0x0070;
constexpr int kWaitLgkm0 = 0xC07F;

// Inline reads of a staging buffer (the momentum variants, where plain loads would raise
// their registers): opaque to the compiler's wait insertion, so no wait for the block
// loading into the other buffer is added; the staged data is known to be complete from the
// wait and barrier that open each block. N reads are in flight together, then one wait.
__device__ __forceinline__ uint32_t lds_addr(const unsigned char *p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) unsigned char *)p;
}
__device__ __forceinline__ uint4 to_uint4(const u32x4_t &v) { return make_uint4(v.x, v.y, v.z, v.w); }
template <int N>
__device__ __forceinline__ void lds_read16_n(const unsigned char *const (&p)[N], uint4 (&u)[N]) {
  u32x4_t v[N > 4 ? 8 : 4];
  if constexpr (N == 1) {
    asm volatile("ds_read_b128 %0, %1\n\ts_waitcnt lgkmcnt(0)" : "=v"(v[0]) : "v"(lds_addr(p[0])) : "memory");
  } else if constexpr (N == 2) {
    asm volatile("ds_read_b128 %0, %2\n\tds_read_b128 %1, %3\n\ts_waitcnt lgkmcnt(0)"
                 : "=&v"(v[0]), "=&v"(v[1])
                 : "v"(lds_addr(p[0])), "v"(lds_addr(p[1]))
                 : "memory");
  } else if constexpr (N == 4) {
    asm volatile(
        "ds_read_b128 %0, %4\n\tds_read_b128 %1, %5\n\tds_read_b128 %2, %6\n\tds_read_b128 %3, %7\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3])
        : "v"(lds_addr(p[0])), "v"(lds_addr(p[1])), "v"(lds_addr(p[2])), "v"(lds_addr(p[3]))
        : "memory");
  } else {
    static_assert(N == 8, "1, 2, 4 or 8 reads");
    asm volatile(
        "ds_read_b128 %0, %8\n\tds_read_b128 %1, %9\n\tds_read_b128 %2, %10\n\tds_read_b128 %3, %11\n\t"
        "ds_read_b128 %4, %12\n\tds_read_b128 %5, %13\n\tds_read_b128 %6, %14\n\tds_read_b128 %7, %15\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(v[0]), "=&v"(v[1]), "=&v"(v[2]), "=&v"(v[3]), "=&v"(v[4]), "=&v"(v[5]), "=&v"(v[6]), "=&v"(v[7])
        : "v"(lds_addr(p[0])), "v"(lds_addr(p[1])), "v"(lds_addr(p[2])), "v"(lds_addr(p[3])),
          "v"(lds_addr(p[4])), "v"(lds_addr(p[5])), "v"(lds_addr(p[6])), "v"(lds_addr(p[7]))
        : "memory");
  }
#pragma unroll
  for (int j = 0; j < N; j++) u[j] = to_uint4(v[j]);
}
__device__ __forceinline__ uint4 lds_read16(const unsigned char *p) {
  const u32x4_t v = *reinterpret_cast<const __attribute__((address_space(3))) u32x4_t *>(
      (const __attribute__((address_space(3))) unsigned char *)p);
  return to_uint4(v);
}
__device__ __forceinline__ void lds_write16(unsigned char *p, uint4 u) {
  *reinterpret_cast<__attribute__((address_space(3))) u32x4_t *>(
      (__attribute__((address_space(3))) unsigned char *)p) = u32x4_t{u.x, u.y, u.z, u.w};
}

constexpr int kZRowSlots = kZMaxBlockRows * kZWaves;   // row partials of one block: [row][wave in group]


// Cross-lane moves of doubles without LDS: DPP within 16-lane rows (quad permutes, half
// and full row mirrors) and the gfx950 lane-half swaps. Each reduction step adds two
// partials that both lanes of a pair add in the same order: results are deterministic.
constexpr int kDppXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kDppXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kDppHalfMirror = 0x141; // lane i <-> 7 - i within each 8 lanes
constexpr int kDppMirror = 0x140;     // lane i <-> 15 - i within each 16 lanes
template <int CTRL>
__device__ __forceinline__ double dpp_d(double x) {
  // every lane reads a defined source lane under these patterns: no old value is needed
  const int lo = __builtin_amdgcn_mov_dpp(__double2loint(x), CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_mov_dpp(__double2hiint(x), CTRL, 0xF, 0xF, false);
  return __hiloint2double(hi, lo);
}
// a, b -> lanes < 32: a[l] + a[l + 32]; lanes >= 32: b[l - 32] + b[l]
__device__ __forceinline__ double swap32_add(double a, double b) {
  const auto lo = __builtin_amdgcn_permlane32_swap(__double2loint(a), __double2loint(b), false, false);
  const auto hi = __builtin_amdgcn_permlane32_swap(__double2hiint(a), __double2hiint(b), false, false);
  return __hiloint2double(hi[0], lo[0]) + __hiloint2double(hi[1], lo[1]);
}
// a, b -> 16-lane rows 0, 2: a summed with the next row; rows 1, 3: b summed with the previous
__device__ __forceinline__ double swap16_add(double a, double b) {
  const auto lo = __builtin_amdgcn_permlane16_swap(__double2loint(a), __double2loint(b), false, false);
  const auto hi = __builtin_amdgcn_permlane16_swap(__double2hiint(a), __double2hiint(b), false, false);
  return __hiloint2double(hi[0], lo[0]) + __hiloint2double(hi[1], lo[1]);
}
// Sums over the wave of RB values per lane (one per row), transposed: the lane halves and
// quarters exchange different rows first. Row b's total ends in lanes [b * 64/RB, (b + 1) * 64/RB).
template <int RB>
__device__ __forceinline__ double wave_sum_rows(const double (&v)[RB]) {
  const int lane = threadIdx.x & 63;
  double x;
  if constexpr (RB == 1) {
    const double w = swap32_add(v[0], v[0]);
    x = swap16_add(w, w);
  } else if constexpr (RB == 2) {
    const double w = swap32_add(v[0], v[1]);
    x = swap16_add(w, w);
  } else if constexpr (RB == 4) {
    x = swap16_add(swap32_add(v[0], v[2]), swap32_add(v[1], v[3]));
  } else {
    static_assert(RB == 8, "1, 2, 4 or 8 rows");
    const double u0 = swap16_add(swap32_add(v[0], v[4]), swap32_add(v[2], v[6]));
    const double u1 = swap16_add(swap32_add(v[1], v[5]), swap32_add(v[3], v[7]));
    const double a = u0 + dpp_d<kDppMirror>(u0), b = u1 + dpp_d<kDppMirror>(u1);
    x = (lane & 8) ? b : a;
  }
  x += dpp_d<kDppXor1>(x);
  x += dpp_d<kDppXor2>(x);
  x += dpp_d<kDppHalfMirror>(x);
  if constexpr (RB < 8) x += dpp_d<kDppMirror>(x);
  return x;
}
// exact (float)(x / d) for double x >= 0 and d > 0 with rd = RN(1 / d): the quotient is
// correctly rounded in double (Markstein) before the rounding to float
__device__ __forceinline__ float div_to_float(double x, double d, double rd) {
  const double q0 = x * rd;
  const double q = fma(fma(-q0, d, x), rd, q0);
  // an infinite (or NaN) sum is its own quotient; the correction would turn inf into NaN
  return (float)(__builtin_isfinite(q0) ? q : q0);
}
// 1 / x and 1 / sqrt(x) to about 2^-50 (hardware estimate and one Newton step)
__device__ __forceinline__ double rcp_d(double x) {
  const double y = __builtin_amdgcn_rcp(x);
  return fma(y, fma(-x, y, 1.0), y);
}
__device__ __forceinline__ double rsq_d(double x) {
  const double y = __builtin_amdgcn_rsq(x);
  return y * fma(-0.5 * x * y, y, 1.5);
}

template <int NSEG, int RB, bool MOM, bool VEC, bool GN, int FIXED = 0>
__device__ __forceinline__ void p1z_body(const DevTensor &t, int band, const StepConsts &k, int mode,
                                         unsigned char *bufA, unsigned char *bufB, float *rbA, float *rbB,
                                         double *rowsh, double *sh, float *rstash) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), lane = threadIdx.x & 63;
  const int64_t m = t.m, ld = t.ld;
  const int zcw = t.zcw;
  // Register staging (aligned rows, no momentum, up to two chunks per wave; the normal step
  // or a gradient-norm pass with its mode fixed at compile time): each wave loads its own
  // pieces of the next block straight into registers by buffer loads while it sums the
  // current one. Lanes past the row's end and rows past the band's end take an offset beyond
  // the buffer's range, so the hardware returns zeros for them. The planner keeps a block's
  // byte span below 2^31 for these tensors.
  constexpr bool REG = VEC && !MOM && NSEG <= 2 && (!GN || FIXED != 0);
  const int wpr = (zcw + NSEG - 1) / NSEG;   // waves per row
  const int grp = wave / wpr;
  const int wg = wave - grp * wpr;           // wave within the group
  const int rpi = t.zrpi;
  constexpr int rb = RB;                     // rows per group and block
  const int br = rpi * rb;                   // rows per block
  const bool active = grp < rpi;
  const int grp_c = active ? grp : 0;        // idle waves read (and discard) group 0's rows
  int P = 1;                                 // wpr rounded up to a power of two
  while (P < wpr) P <<= 1;
  bool sok[NSEG];
  int chs[NSEG];
  int64_t col[NSEG];
#pragma unroll
  for (int s = 0; s < NSEG; s++) {
    chs[s] = wg + s * wpr;
    col[s] = (int64_t)chs[s] * kChunk + lane * 8;
    sok[s] = active && chs[s] < zcw && col[s] < m;
  }
  const int64_t r0 = (int64_t)band * t.zrows;
  const int64_t r1 = (t.n - r0 < t.zrows) ? t.n : r0 + t.zrows;
  const int64_t nblk = (r1 - r0 + br - 1) / br;
  const int npieces = br * zcw;          // 1 KiB pieces of gradient per block
  const int goff_m = npieces * 1024;     // momentum pieces follow (2 KiB each)
  const float sc = MOM ? k.s_m : k.s_0;
  const float deps = sqrtf(k.eps);                  // the oracle's D on the floor
  const float reps = (float)(1.0 / (double)deps);   // correctly rounded 1/D
  const double dm = (double)m, rdm = 1.0 / dm;
  // the sums this step forms (the clip stage's prediction from the last step)
  const int regime = __builtin_amdgcn_readfirstlane(ldg(&t.sc->regime));
  const bool want_z = regime != kRegimeFloor, want_y = regime != kRegimeAbove;

  double cacc[NSEG][8], zacc[NSEG][8];
#pragma unroll
  for (int s = 0; s < NSEG; s++)
#pragma unroll
    for (int e = 0; e < 8; e++) cacc[s][e] = zacc[s][e] = 0.0;
  double ysum = 0.0, ysum2 = 0.0, umax = 0.0;   // the floored sum in two chains
  // mode 1 (sums only): the band's sum of g^2, kept by lane b * P of each group's first wave
  double rs_l = 0.0;
  // mode 2: the gradient scale of the gradient-norm mode (elements enter as fl(c g))
  const bool scaled = mode == 2;
  const float gc = scaled ? ldg(k.gscale) : 1.f;
  // a row with R_i == 0 but a nonzero sum (flagged by lane b * P of the group's first wave)
  int bad_l = 0;

  // Block loads: piece p = (row r, chunk c) of the block goes to wave p % 8. Rows past
  // the band's end and lanes past the row's end load zeros (from a zero block in global
  // memory), so they add nothing to any sum and the sweeps need no masks. Wave 0 also
  // stages the block's old R values.
  const int pr0 = wave / zcw, pc0 = wave - pr0 * zcw;                   // piece `wave`: (row, chunk)
  const int dr = kZWaves / zcw, dc = kZWaves - (kZWaves / zcw) * zcw;   // step of 8 pieces
  // Direct loads (the lean loop): the lane's source moves by a fixed step from piece to
  // piece, and bit c of cmask says whether its 8 columns of chunk c lie in the row (zcw <= 32:
  // at most 8 waves of 4 chunks). The base pointers are held in registers for the whole band
  // (read once, not per piece). With momentum, the fp32 row of M follows in two 1 KiB halves
  // per piece (masks cm0, cm1). The momentum variants with four chunks per wave or in the
  // gradient-norm passes keep the general loop: the registers of the lean one would spill.
  constexpr bool LEAN = !REG && VEC && (!MOM || (NSEG <= 2 && !GN));
  uint32_t cmask = 0, cm0 = 0, cm1 = 0;
  const uint16_t *gptr = t.g, *zptr = t.zeros;
  const float *mptr = t.M, *rptr = t.R;
  if constexpr (LEAN) {
    for (int c = 0; c < zcw; c++) {
      if ((int64_t)c * kChunk + lane * 8 < m) cmask |= 1u << c;
      if ((int64_t)c * kChunk + lane * 4 < m) cm0 |= 1u << c;
      if ((int64_t)c * kChunk + lane * 4 + 256 < m) cm1 |= 1u << c;
    }
    asm volatile("" : "+v"(gptr), "+v"(zptr), "+v"(rptr));
    if constexpr (MOM) asm volatile("" : "+v"(mptr));
  }
  const int64_t off_step = (int64_t)dr * ld + (int64_t)dc * kChunk;
  const int64_t off_wrap = ld - (int64_t)zcw * kChunk;
  auto issue = [&](int64_t blk, unsigned char *buf, float *rbuf) {
    const int64_t rbase = r0 + blk * br;
    int r = pr0, c = pc0;
    if constexpr (LEAN) {
      int64_t off = (rbase + pr0) * ld + (int64_t)pc0 * kChunk + lane * 8;   // elements of G
      int64_t moff = (rbase + pr0) * m + (int64_t)pc0 * kChunk + lane * 4;   // elements of M
      for (int p = wave; p < npieces; p += kZWaves) {
        const bool rok = rbase + r < r1;
        dma16((rok && ((cmask >> c) & 1u)) ? (const void *)(gptr + off) : (const void *)zptr,
              buf + (size_t)p * 1024);
        if constexpr (MOM) {
          dma16((rok && ((cm0 >> c) & 1u)) ? (const void *)(mptr + moff) : (const void *)zptr,
                buf + goff_m + (size_t)p * 2048);
          dma16((rok && ((cm1 >> c) & 1u)) ? (const void *)(mptr + moff + 256) : (const void *)zptr,
                buf + goff_m + (size_t)p * 2048 + 1024);
          moff += (int64_t)dr * m + (int64_t)dc * kChunk;
        }
        r += dr;
        c += dc;
        off += off_step;
        if (c >= zcw) {
          c -= zcw;
          r++;
          off += off_wrap;
          if constexpr (MOM) moff += m - (int64_t)zcw * kChunk;
        }
      }
    } else
    for (int p = wave; p < npieces; p += kZWaves) {
      const bool rok = rbase + r < r1;   // wave-uniform
      const int64_t i = rok ? rbase + r : r1 - 1;
      const int64_t cg = (int64_t)c * kChunk + lane * 8;
      if (VEC) {
        dma16((rok && cg < m) ? (const void *)(t.g + i * ld + cg) : (const void *)t.zeros, buf + (size_t)p * 1024);
      } else {
        lds_write16(buf + (size_t)p * 1024 + lane * 16, rok ? load_bf8(t.g, ld, m, i, cg) : make_uint4(0u, 0u, 0u, 0u));
      }
      if (MOM) {
        const float *mrow = t.M + i * m;
        const int64_t c0 = (int64_t)c * kChunk + lane * 4, c1 = c0 + 256;
        if (VEC) {
          dma16((rok && c0 < m) ? (const void *)(mrow + c0) : (const void *)t.zeros, buf + goff_m + (size_t)p * 2048);
          dma16((rok && c1 < m) ? (const void *)(mrow + c1) : (const void *)t.zeros,
                buf + goff_m + (size_t)p * 2048 + 1024);
        } else {
          uint32_t mv[8];
#pragma unroll
          for (int e = 0; e < 4; e++) {
            mv[e] = (rok && c0 + e < m) ? __float_as_uint(ldg(mrow + c0 + e)) : 0u;
            mv[4 + e] = (rok && c1 + e < m) ? __float_as_uint(ldg(mrow + c1 + e)) : 0u;
          }
          lds_write16(buf + goff_m + (size_t)p * 2048 + lane * 16, make_uint4(mv[0], mv[1], mv[2], mv[3]));
          lds_write16(buf + goff_m + (size_t)p * 2048 + 1024 + lane * 16, make_uint4(mv[4], mv[5], mv[6], mv[7]));
        }
      }
      r += dr;
      c += dc;
      if (c >= zcw) {
        c -= zcw;
        r++;
      }
    }
    if (wave == 0) {
      const int64_t i = rbase + (lane < br ? lane : br - 1);
      const int64_t ic = i < r1 ? i : r1 - 1;
      if (LEAN)
        dma4(rptr + ic, rbuf);
      else if (VEC)
        dma4(t.R + ic, rbuf);
      else
        rbuf[lane] = ldg(t.R + ic);
    }
  };
  // register staging: byte offsets of the lane's pieces from the block's first row (the
  // sentinel 2^31 lies beyond any block's range), the block's buffer descriptor, and the old
  // R of the row whose fold the lane takes part in (lane b * P + w: row b of its group)
  uint32_t vo[RB][NSEG];
  const int rfold = grp_c * RB + ((lane / P) < RB ? (lane / P) : 0);
  if constexpr (REG) {
#pragma unroll
    for (int b = 0; b < RB; b++)
#pragma unroll
      for (int s = 0; s < NSEG; s++)
        vo[b][s] = sok[s] ? (uint32_t)((((int64_t)grp_c * RB + b) * ld + col[s]) * 2) : 0x80000000u;
  }
  auto issue_reg = [&](int64_t blk, u32x4_t (&dst)[RB][NSEG], float &rold) {
    const int64_t rbase = r0 + blk * br;
    const int64_t span = (r1 - rbase) * ld * 2;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(t.g + rbase * ld), (short)0, (int)(span < 0x7FFFFFFF ? span : 0x7FFFFFFF), 0x00020000);
#pragma unroll
    for (int b = 0; b < RB; b++)
#pragma unroll
      for (int s = 0; s < NSEG; s++) {
        dst[b][s] = __builtin_amdgcn_raw_buffer_load_b128(rs, vo[b][s], 0, 0);
      }
    const int64_t i = rbase + rfold;
    rold = ldg(t.R + (i < r1 ? i : r1 - 1));
  };
  // The lane's NSEG pieces of RB block rows are read from LDS in batches of RBB rows into
  // uk[b0 .. b0 + RBB). Staged padding is zero; a segment past the row's last chunk
  // (wave-uniform) reads the buffer's zero area instead. Every address lies in the buffer
  // being read, which the compiler can tell from the one the next block is loading into,
  // so plain reads wait for the LDS alone (lgkmcnt), never for that load. The momentum
  // variants keep one inline batch with its wait: plain reads there raise the registers
  // the compiler holds (and spills).
  constexpr int RBB = (8 / NSEG < RB ? 8 / NSEG : RB) > 0 ? (8 / NSEG < RB ? 8 / NSEG : RB) : 1;
  // the block's staged gradient stays in registers from the first sweep to the second where
  // it fits (no momentum, up to three chunks per wave; the other variants would spill)
  constexpr bool KEEP = !MOM && NSEG <= 3;
  auto read_rows = [&](const unsigned char *buf, int b0, uint4 (&uk)[RB][NSEG]) {
    const unsigned char *ptr[RBB * NSEG];
#pragma unroll
    for (int b = 0; b < RBB; b++)
#pragma unroll
      for (int s = 0; s < NSEG; s++)
        ptr[b * NSEG + s] =
            buf + (chs[s] < zcw ? (size_t)((grp_c * RB + b0 + b) * zcw + chs[s]) * 1024 : (size_t)kZLdsBytes) +
            lane * 16;
    if constexpr (KEEP) {
#pragma unroll
      for (int b = 0; b < RBB; b++)
#pragma unroll
        for (int s = 0; s < NSEG; s++) uk[b0 + b][s] = lds_read16(ptr[b * NSEG + s]);
    } else {
      uint4 u[RBB * NSEG];
      lds_read16_n<RBB * NSEG>(ptr, u);
#pragma unroll
      for (int b = 0; b < RBB; b++)
#pragma unroll
        for (int s = 0; s < NSEG; s++) uk[b0 + b][s] = u[b * NSEG + s];
    }
  };
  auto step = [&](int64_t blk, unsigned char *cur, float *rcur, unsigned char *nxt, float *rnxt,
                  u32x4_t (&regc)[RB][NSEG], float rold, u32x4_t (&regn)[RB][NSEG], float &rnold, auto zc, auto yc) {
    if constexpr (REG) {
      // the next block's loads go out first; the compiler waits for this block's registers
      // where they are first used
      if (blk + 1 < nblk) issue_reg(blk + 1, regn, rnold);
    } else {
      __builtin_amdgcn_s_waitcnt(kWaitVmLgkm0);   // this block's loads (issued one block earlier)
      __builtin_amdgcn_s_barrier();               // ... by every wave; the other buffer is free
      if (blk + 1 < nblk) issue(blk + 1, nxt, rnxt);
    }
    const int64_t rbase = r0 + blk * br;
    double *slot = rowsh + (blk & 1) * kZRowSlots;   // [block row][wave in group]
    // the lane's staged gradient of the block (the second sweep reads it again unless KEEP)
    uint4 uk[RB][NSEG];
    // row and column sums of g^2 (bf16 squares are exact in double); an idle wave's
    // accumulators are never used. Mode 2 has them from the first pass.
    if (mode != 2) {
      double rp[RB];
#pragma unroll
      for (int b0 = 0; b0 < RB; b0 += RBB) {
        if constexpr (REG) {
#pragma unroll
          for (int bb = 0; bb < RBB; bb++)
#pragma unroll
            for (int s = 0; s < NSEG; s++) uk[b0 + bb][s] = to_uint4(regc[b0 + bb][s]);
        } else {
          read_rows(cur, b0, uk);
        }
#pragma unroll
        for (int bb = 0; bb < RBB; bb++) {
          const int b = b0 + bb;
          double ra = 0.0, rb2 = 0.0;   // two chains per row
#pragma unroll
          for (int s = 0; s < NSEG; s++) {
            // one 8-element group at a time (the scheduler would otherwise convert every
            // staged element to double at once)
            __builtin_amdgcn_sched_barrier(0);
            float x[8];
            unpack8(uk[b][s], x);
#pragma unroll
            for (int e = 0; e < 8; e++) {
              const double xd = (double)x[e];
              if (e & 1)
                rb2 = fma(xd, xd, rb2);
              else
                ra = fma(xd, xd, ra);
              cacc[s][e] = fma(xd, xd, cacc[s][e]);
            }
            // the column sums are formed here, not sunk towards the loop's end (which
            // would keep every converted element live across the block)
#pragma unroll
            for (int e = 0; e < 8; e++) asm volatile("" : "+v"(cacc[s][e]));
          }
          rp[b] = ra + rb2;
        }
      }
      __builtin_amdgcn_sched_barrier(0);
      const double rsum = wave_sum_rows<RB>(rp);
      if (active && (lane & (64 / RB - 1)) == 0) slot[(grp * RB + lane / (64 / RB)) * kZWaves + wg] = rsum;
    }
    __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
    __builtin_amdgcn_s_barrier();
    // R_i after the EMA (Eq. 1) for the group's rb rows, lane-parallel: lane b * P + w
    // takes the partial of wave w of row b; after the segment sum lane b * P holds the row
    double winv_l = 0.0;
    if (mode == 2) {
      // R_i folded this step (staged with the block)
      const int b = lane / P, w = lane - b * P;
      const int r = grp_c * rb + (b < rb ? b : 0);
      const int64_t i = rbase + r;
      const float R = REG ? rold : rcur[r];   // (REG: the folded R of the lane's row r)
      const double Rd = (double)R;
      const bool normal = R > 0.f && R < __builtin_inff();
      winv_l = (normal && i < r1) ? rcp_d(Rd) : 0.0;   // (1/R is 0 for R = +inf)
      if (active && wg == 0 && b < rb && w == 0 && i < r1) {
        rstash[i - r0] = R;
        if (R != R) bad_l = 1;
      }
    } else {
      const int b = lane / P, w = lane - b * P;
      const int r = grp_c * rb + (b < rb ? b : 0);
      double x = (active && b < rb && w < wpr) ? slot[r * kZWaves + w] : 0.0;
      if (P >= 2) x += dpp_d<kDppXor1>(x);
      if (P >= 4) x += dpp_d<kDppXor2>(x);
      if (P >= 8) x += dpp_d<kDppHalfMirror>(x);
      const int64_t i = rbase + r;
      if (mode == 1) {
        // the row's sum of g^2: R is folded once the gradient scale is known
        if (active && wg == 0 && b < rb && w == 0 && i < r1) {
          stg(t.ainv + i, x);
          rs_l += x;
        }
      } else {
      const float ri = div_to_float(x, dm, rdm);
      const float Rold = REG ? rold : rcur[r];   // (REG: the lane's row is r)
      const float R = fmaf(k.a2, ri, __fmul_rn(k.b2, Rold));
      const double Rd = (double)R;
      const bool normal = R > 0.f && R < __builtin_inff();
      winv_l = (normal && i < r1) ? rcp_d(Rd) : 0.0;   // (1/R is 0 for R = +inf)
      if (active && wg == 0 && b < rb && w == 0 && i < r1) {
        // staged for the band's end: a global store here would hold up the next block's
        // wait for its staged rows until the store completes
        rstash[i - r0] = R;
        if (R != R || (!(R > 0.f) && x > 0.0)) bad_l = 1;
      }
      }
    }
    // z_j, the floored sum and the bound (the sums the prediction asks for)
    auto sweep2 = [&](auto zc, auto yc) {
      constexpr bool Z = decltype(zc)::value, Y = decltype(yc)::value;
#pragma unroll
      for (int b0 = 0; b0 < RB; b0 += RBB) {
      if constexpr (!REG) {
        if (!KEEP || mode == 2) read_rows(cur, b0, uk);   // (mode 2: the first sweep did not run)
      } else {
        // the packed block is unpacked again here, from its own registers (not needed after
        // this sweep, so the empty asm may claim to change them: no copy is made); keeping
        // sweep 1's floats beside the next block's registers would spill
#pragma unroll
        for (int bb = 0; bb < RBB; bb++)
#pragma unroll
          for (int s = 0; s < NSEG; s++) {
            asm volatile("" : "+v"(regc[b0 + bb][s]));
            uk[b0 + bb][s] = to_uint4(regc[b0 + bb][s]);
          }
      }
#pragma unroll
      for (int bb = 0; bb < RBB; bb++) {
        const int b = b0 + bb;
        const int r = grp_c * rb + b;
        const int src = b * P;
        const double winv = __hiloint2double(__builtin_amdgcn_readlane(__double2hiint(winv_l), src),
                                             __builtin_amdgcn_readlane(__double2loint(winv_l), src));
        float amax = 0.f;   // max |s x| over the lane's elements of the row
#pragma unroll
        for (int s = 0; s < NSEG; s++) {
          // one 8-element group at a time where the block is read from LDS here; with the
          // block in registers the scheduler may interleave the groups (1% faster, no spills)
          if constexpr (!KEEP) __builtin_amdgcn_sched_barrier(0);
          float x[8];
          unpack8(uk[b][s], x);
          if (scaled) {
#pragma unroll
            for (int e = 0; e < 8; e++) x[e] = gc * x[e];
          }
          if (MOM) {
            const unsigned char *mp =
                cur + (chs[s] < zcw ? goff_m + (size_t)(r * zcw + chs[s]) * 2048 : (size_t)kZLdsBytes) + lane * 32;
            const unsigned char *mpp[2] = {mp, mp + 16};
            uint4 mv[2];
            lds_read16_n<2>(mpp, mv);
            const float mo[8] = {__uint_as_float(mv[0].x), __uint_as_float(mv[0].y), __uint_as_float(mv[0].z),
                                 __uint_as_float(mv[0].w), __uint_as_float(mv[1].x), __uint_as_float(mv[1].y),
                                 __uint_as_float(mv[1].z), __uint_as_float(mv[1].w)};
#pragma unroll
            for (int e = 0; e < 8; e++) x[e] = fmaf(k.a1, x[e], __fmul_rn(k.b1, mo[e]));
          }
#pragma unroll
          for (int e = 0; e < 8; e++) {
            const float ax = __fmul_rn(sc, x[e]);
            if (Z) {
              const double axd = (double)ax;
              zacc[s][e] = fma(axd * axd, winv, zacc[s][e]);
              amax = fmaxf(amax, fabsf(ax));
            }
            if (Y) {
              const float q0 = ax * reps;
              const float uf = fmaf(fmaf(-q0, deps, ax), reps, q0);   // RN(ax / deps)
              if (e & 1)
                ysum2 = fma((double)uf, (double)uf, ysum2);
              else
                ysum = fma((double)uf, (double)uf, ysum);
            }
          }
        }
        if (Z) umax = fmax(umax, ((double)amax * (double)amax) * winv);
        // a row with R_i == 0 but nonzero elements (mode 0 tests its sum instead)
        if (Z && scaled && winv == 0.0 && amax > 0.f) bad_l = 1;
      }
      }
      __builtin_amdgcn_sched_barrier(0);
    };
    // an idle wave (its rows are group 0's) adds nothing; mode 1 forms no update sums
    if (active && mode != 1) sweep2(zc, yc);
  };
  u32x4_t regA[RB][NSEG], regB[RB][NSEG];
  float roldA = 0.f, roldB = 0.f;
  if constexpr (REG)
    issue_reg(0, regA, roldA);
  else
    issue(0, bufA, rbA);
  // the band's loop, specialised for the sums it forms (the regime is the same for the band)
  auto band_loop = [&](auto zc, auto yc) {
    for (int64_t blk = 0; blk < nblk; blk += 2) {
      step(blk, bufA, rbA, bufB, rbB, regA, roldA, regB, roldB, zc, yc);
      if (blk + 1 >= nblk) break;
      step(blk + 1, bufB, rbB, bufA, rbA, regB, roldB, regA, roldA, zc, yc);
    }
  };
  if (want_z && want_y)
    band_loop(std::true_type(), std::true_type());
  else if (want_z)
    band_loop(std::true_type(), std::false_type());
  else
    band_loop(std::false_type(), std::true_type());
  __builtin_amdgcn_s_waitcnt(kWaitVmLgkm0);
  __syncthreads();
  // column partials: groups 1.. add theirs into group 0's through LDS, in group order
  double *colbuf = reinterpret_cast<double *>(bufA);   // zcw * 512 doubles: groups > 1 only when zcw <= 8
  for (int gsrc = 1; gsrc < rpi; gsrc++) {
#pragma unroll
    for (int half = 0; half < 2; half++) {
      if (grp == gsrc) {
#pragma unroll
        for (int s = 0; s < NSEG; s++)
          if (chs[s] < zcw)
#pragma unroll
            for (int e = 0; e < 8; e++) colbuf[chs[s] * kChunk + lane * 8 + e] = half ? zacc[s][e] : cacc[s][e];
      }
      __syncthreads();
      if (grp == 0) {
#pragma unroll
        for (int s = 0; s < NSEG; s++)
          if (chs[s] < zcw)
#pragma unroll
            for (int e = 0; e < 8; e++) {
              const double v = colbuf[chs[s] * kChunk + lane * 8 + e];
              if (half) zacc[s][e] += v; else cacc[s][e] += v;
            }
      }
      __syncthreads();
    }
  }
  if (grp == 0) {
    const int64_t prow = (int64_t)band * m;
#pragma unroll
    for (int s = 0; s < NSEG; s++) {
      if (!sok[s]) continue;
#pragma unroll
      for (int e = 0; e < 8; e++) {
        if (VEC || col[s] + e < m) {
          if (mode != 2) stg(t.colpart + prow + col[s] + e, cacc[s][e]);
          if (mode != 1) stg(t.zpart + prow + col[s] + e, zacc[s][e]);
        }
      }
    }
  }
  // the band's R and 1/sqrt(R) (coalesced), and its statistics: fixed-order reductions
  // (mode 1: the band's sum of g^2 instead; mode 2: R was written by the fold)
  const int64_t nrows = r1 - r0;
  double rs = rs_l, rdup = 0.0;
  float rmn = __builtin_inff(), rmx = 0.f;
  for (int64_t j = threadIdx.x; mode != 1 && j < nrows; j += kZThreads) {
    const float R = rstash[j];
    if (j > 0 && R > 0.f && R == rstash[j - 1]) rdup += 1.0;
    const double Rd = (double)R;
    const bool normal = R > 0.f && R < __builtin_inff();
    if (mode == 0) {
      stg(t.R + r0 + j, R);
      stg(t.ainv + r0 + j, normal ? rsq_d(Rd) : 1.0 / sqrt(Rd));
    }
    rs += Rd;
    if (R > 0.f) rmn = fminf(rmn, R);
    rmx = fmaxf(rmx, R);
  }
  const double ys = wg_sum_w<kZWaves>(ysum + ysum2, sh);
  const double um = wg_max_w<kZWaves>(umax, sh);
  const double rsum = wg_sum_w<kZWaves>(rs, sh);
  const float rmin = wg_min_wf<kZWaves>(rmn, sh);
  const float rmax = wg_max_wf<kZWaves>(rmx, sh);
  const int bd = wg_or_w<kZWaves>(bad_l, sh);
  const double rd = wg_sum_w<kZWaves>(rdup, sh);
  if (threadIdx.x == 0) {
    stg(&t.bst[band].rdup, (int32_t)rd);
    stg(&t.bst[band].rsum, rsum);
    stg(&t.bst[band].ysum, ys);
    stg(&t.bst[band].umax, um);
    stg(&t.bst[band].rmin, rmin);
    stg(&t.bst[band].rmax, rmax);
    stg(&t.bst[band].bad, bd);
    stg(&t.bst[band].regime, (int32_t)regime);
  }
}

// GN: the gradient-norm mode's passes (mode 1, the sums of g^2 alone, or mode 2, z and the
// floored sum of the scaled gradient once R is folded); without it the mode is 0 at compile
// time. FIXED: one of those passes (1 or 2) with its mode fixed at compile time, staged in
// registers.
template <int NSEG, bool MOM, bool VEC, bool GN, int FIXED = 0>
__global__ __launch_bounds__(kZThreads) void p1z_kernel(const DevTensor *__restrict__ TT,
                                                        const Item *__restrict__ items, StepConsts k, int mode_arg) {
  __shared__ __attribute__((aligned(16))) unsigned char bufA[kZLdsBytes + 2048];
  __shared__ __attribute__((aligned(16))) unsigned char bufB[kZLdsBytes + 2048];
  __shared__ float rbA[64], rbB[64];
  __shared__ double rowsh[2 * kZRowSlots];
  __shared__ double sh[5 * kZWaves];
  __shared__ float rstash[kZMaxBandRows];
  // each buffer ends in a zero area of 32 bytes per lane, cleared before the first block's wait
  reinterpret_cast<uint32_t *>(bufA + kZLdsBytes)[threadIdx.x] = 0u;
  reinterpret_cast<uint32_t *>(bufB + kZLdsBytes)[threadIdx.x] = 0u;
  static_assert(kZThreads * 4 == 2048, "one word per thread");
  const int mode = FIXED != 0 ? FIXED : GN ? mode_arg : 0;
  const Item it = items[blockIdx.x];
  const DevTensor &t = TT[it.tensor];
  // rows per group and block: the planner keeps 4 at most with one or two chunks per wave,
  // 2 with three and 1 with four, which keeps every variant's loop free of register spills
  // (the gradient-norm mode's register-staged z pass takes 2: with 4 its registers spill)
  constexpr int RB4 = FIXED == 2 ? 2 : 4;
  if (NSEG <= 2 && t.zrb >= 4)
    p1z_body<NSEG, NSEG <= 2 ? RB4 : 1, MOM, VEC, GN, FIXED>(t, it.tile, k, mode, bufA, bufB, rbA, rbB, rowsh, sh, rstash);
  else if (NSEG <= 3 && t.zrb >= 2)
    p1z_body<NSEG, NSEG <= 3 ? 2 : 1, MOM, VEC, GN, FIXED>(t, it.tile, k, mode, bufA, bufB, rbA, rbB, rowsh, sh, rstash);
  else
    p1z_body<NSEG, 1, MOM, VEC, GN, FIXED>(t, it.tile, k, mode, bufA, bufB, rbA, rbB, rowsh, sh, rstash);
}

// Reductions of the clip stage, over the whole work-group (a tensor of its own) or over one
// wave (the slices of a stacked tensor, one slice per wave at a time). Every participating
// lane gets the result, in a fixed order.
struct RedGroup {
  double *sh;
  static constexpr int kN = kThreads;
  __device__ __forceinline__ int lane() const { return (int)threadIdx.x; }
  __device__ __forceinline__ bool lead() const { return threadIdx.x == 0; }
  __device__ __forceinline__ double sum(double x) const { return block_sum(x, sh); }
  __device__ __forceinline__ double max(double x) const { return wg_max_w<kWaves>(x, sh); }
  __device__ __forceinline__ float minf(float x) const { return wg_min_wf<kWaves>(x, sh); }
  __device__ __forceinline__ float maxf(float x) const { return wg_max_wf<kWaves>(x, sh); }
  __device__ __forceinline__ int any(int x) const { return wg_or_w<kWaves>(x, sh); }
};
struct RedWave {
  static constexpr int kN = 64;
  __device__ __forceinline__ int lane() const { return (int)(threadIdx.x & 63); }
  __device__ __forceinline__ bool lead() const { return (threadIdx.x & 63) == 0; }
  __device__ __forceinline__ double sum(double x) const { return wave_sum_d(x); }
  __device__ __forceinline__ double max(double x) const { return wave_max_d(x); }
  __device__ __forceinline__ float minf(float x) const { return wave_min_f(x); }
  __device__ __forceinline__ float maxf(float x) const { return wave_max_f(x); }
  __device__ __forceinline__ int any(int x) const { return wave_or(x); }
};
template <class Red>
__device__ __forceinline__ double red_sum(const Red &r, const double *p, int64_t n, int64_t stride = 1) {
  double s = 0.0;
  for (int64_t c = r.lane(); c < n; c += Red::kN) s += ldg(p + c * stride);
  return r.sum(s);
}

// fixed-order work-group sum of p[0], p[stride], ..., p[(n-1) stride]: thread j sums
// entries j, j + 256, ..., then a tree; every thread of the (256-thread) work-group calls it
__device__ __forceinline__ double wg_sum(const double *p, int64_t n, double *sh, int64_t stride = 1) {
  double s = 0.0;
  for (int64_t c = threadIdx.x; c < n; c += kThreads) s += ldg(p + c * stride);
  return block_sum(s, sh);
}
// q = max(mean R, eps) for a factored tensor (the clamp of the reconstruction), from the
// sums of R over the fold chunks of rows or over the row bands
template <class Red>
__device__ __forceinline__ float mean_r_of(const DevTensor &t, const StepConsts &k, const Red &r) {
  // row-band tensors keep the sums of R in their band statistics, except in the gradient-
  // norm mode, where the fold forms R and its sums per chunk of rows as for wide tensors
  const double sr = (t.zpath && !k.gclip) ? red_sum(r, &t.bst->rsum, t.nzb, sizeof(BandStats) / sizeof(double))
                                          : red_sum(r, t.rsum, t.zpath ? (t.n + kFold - 1) / kFold : t.nfr);
  return max_nan((float)(sr / (double)t.n), k.eps);
}
__device__ __forceinline__ float mean_r_clamped(const DevTensor &t, const StepConsts &k, double *sh) {
  return mean_r_of(t, k, RedGroup{sh});
}

// Extremes of the positive values and equal neighbours within one fold chunk (v of this
// thread's row or column, 0 past the end), for the clip stage's test of repeated factors;
// every thread of the work-group calls it
__device__ __forceinline__ void chunk_repeats(ColStats *out, float v, float *nb, double *sh) {
  nb[threadIdx.x] = v;
  __syncthreads();
  const double dup = (threadIdx.x > 0 && v > 0.f && v == nb[threadIdx.x - 1]) ? 1.0 : 0.0;
  const double d = block_sum(dup, sh);
  const float mn = wg_min_wf<kWaves>(v > 0.f ? v : __builtin_inff(), sh);
  const float mx = wg_max_wf<kWaves>(v, sh);
  if (threadIdx.x == 0) {
    stg(&out->cmin, mn);
    stg(&out->cmax, mx);
    stg(&out->cdup, (int32_t)d);
  }
}

// --------------------------------------------------------------------------------------------
// fold: R_i <- b2 R_i + a2 r_i, C_j <- b2 C_j + a2 c_j (Eq. 1), 1/sqrt(R_i), sums of R
// --------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void fold_kernel(const DevTensor *__restrict__ TT,
                                                        const Item *__restrict__ items, StepConsts k, int phase) {
  __shared__ double sh[kThreads];
  const Item it = items[blockIdx.x];
  const DevTensor &t = TT[it.tensor];
  // gradient-norm mode: the statistics of the scaled gradient are c^2 times the exact sums
  const double c2 = phase == 1 ? (double)ldg(k.gscale) * (double)ldg(k.gscale) : 1.0;
  // row chunks of this launch: wide tensors always; row-band tensors only in phase 1,
  // where their row sums of g^2 wait in ainv
  const int nrows = t.zpath ? (phase == 1 ? (int)((t.n + kFold - 1) / kFold) : 0) : t.nfr;
  if (phase == 2 && !t.zpath) return;
  __shared__ float nb[kThreads];
  if (it.tile < nrows) {
    const int64_t i = (int64_t)it.tile * kFold + threadIdx.x;
    double rn = 0.0;
    float Rv = 0.f;
    if (i < t.n) {
      double s = 0.0;
      if (t.zpath)
        s = ldg(t.ainv + i);
      else
#pragma unroll 8
        for (int q = 0; q < t.ntc; q++) s += ldg(t.rowpart + (int64_t)q * t.n + i);
      const float ri = (float)((phase == 1 ? c2 * s : s) / (double)t.m);
      const float R = fmaf(k.a2, ri, __fmul_rn(k.b2, ldg(t.R + i)));
      stg(t.R + i, R);
      stg(t.ainv + i, 1.0 / sqrt((double)R));
      rn = (double)R;
      Rv = R;
    }
    const double tot = block_sum(rn, sh);
    if (threadIdx.x == 0) stg(t.rsum + it.tile, tot);
    if (!t.zpath) chunk_repeats(t.cst + it.tile, Rv, nb, sh);
  } else if (!t.zpath || phase == 1) {
    // C_j from the column partials ([row bands][m] of either pass 1)
    const int64_t j = (int64_t)(it.tile - nrows) * kFold + threadIdx.x;
    float Cv = 0.f;
    if (j < t.m) {
      double s = 0.0;
      const int nb = t.zpath ? t.nzb : t.ntr;
#pragma unroll 8
      for (int b = 0; b < nb; b++) s += ldg(t.colpart + (int64_t)b * t.m + j);
      const float cj = (float)((phase == 1 ? c2 * s : s) / (double)t.n);
      Cv = fmaf(k.a2, cj, __fmul_rn(k.b2, ldg(t.C + j)));
      stg(t.C + j, Cv);
    }
    if (!t.zpath) chunk_repeats(t.cst + t.nfr + (it.tile - nrows), Cv, nb, sh);
  } else {
    // row-band tensor: C_j (phase 0; phase 2 has it from phase 1), c'_j = C_j / max(mean R,
    // eps) and sum_j z_j / c'_j over the chunk
    __shared__ float cprev[kThreads];
    const float q = mean_r_clamped(t, k, sh);
    const int64_t j = (int64_t)it.tile * kFold + threadIdx.x;
    double sj = 0.0, sj2 = 0.0;
    float cmn = __builtin_inff(), cmx = 0.f, Cj = 0.f;
    int bad = 0;
    if (j < t.m) {
      double cs = 0.0, zs = 0.0;
      // loads of several bands in flight; the sums still run in band order
#pragma unroll 8
      for (int p = 0; p < t.nzb; p++) {
        cs += ldg(t.colpart + (int64_t)p * t.m + j);
        zs += ldg(t.zpart + (int64_t)p * t.m + j);
      }
      float C;
      if (phase == 0) {
        const float cj = (float)(cs / (double)t.n);
        C = fmaf(k.a2, cj, __fmul_rn(k.b2, ldg(t.C + j)));
        stg(t.C + j, C);
      } else {
        C = ldg(t.C + j);
      }
      Cj = C;
      const float cp = C / q;
      if (C > 0.f) {
        // c'_j that is zero or not finite leaves the tensor to the exact pass
        if (cp > 0.f && cp < __builtin_inff()) {
          sj = zs / (double)cp;
          sj2 = sj / (double)cp;
          cmn = cmx = cp;
        } else {
          bad = 1;
        }
      } else if (C != 0.f || cs > 0.0 || zs > 0.0) {
        bad = 1;   // NaN, or a nonzero column whose C underflowed
      }
    }
    // repeated column factors: C_j equal to the previous column's (within the chunk)
    cprev[threadIdx.x] = Cj;
    __syncthreads();
    const double dup = (threadIdx.x > 0 && Cj > 0.f && Cj == cprev[threadIdx.x - 1]) ? 1.0 : 0.0;
    const double S = block_sum(sj, sh);
    const double S2 = block_sum(sj2, sh);
    const double cdup = block_sum(dup, sh);
    const float cmin = wg_min_wf<kWaves>(cmn, sh);
    const float cmax = wg_max_wf<kWaves>(cmx, sh);
    const int b = wg_or_w<kWaves>(bad, sh);
    if (threadIdx.x == 0) {
      stg(&t.cst[it.tile].cdup, (int32_t)cdup);
      stg(&t.cst[it.tile].s2, S2);
      stg(&t.cst[it.tile].s, S);
      stg(&t.cst[it.tile].cmin, cmin);
      stg(&t.cst[it.tile].cmax, cmax);
      stg(&t.cst[it.tile].bad, b);
    }
  }
}

// Gradient-norm mode: sum of g^2 of each (tile, part) of an exact tensor, into its update-sum
// slot (the update-sum pass later overwrites it); factored items have theirs in pass 1
__global__ __launch_bounds__(kThreads) void gsq_kernel(const DevTensor *__restrict__ TT,
                                                       const Item *__restrict__ items) {
  __shared__ double sh[kThreads];
  const Item it = items[blockIdx.x];   // it.tile = tile * kSub + part
  const DevTensor &t = TT[it.tensor];
  if (t.kind == kFactored) return;
  const Tile tl = tile_of(t, it.tile / kSub);
  const WaveMap wm(t, tl);
  const int64_t r0 = wm.wr + (int64_t)(it.tile % kSub) * wm.rpi, rs = (int64_t)wm.rpi * kSub;
  double acc = 0.0;
  for (int64_t lr = r0; lr < tl.nr; lr += rs) {
    const int64_t i = tl.row(lr);
#pragma unroll
    for (int e = 0; e < 8; e++) {
      if (wm.col + e >= t.m) continue;
      const double g = (double)elem(t.g, i * t.ld + wm.col + e, t.fp32);
      acc += g * g;
    }
  }
  const double s = block_sum(acc, sh);
  if (threadIdx.x == 0) stg(t.ssum + it.tile, s);
}

// Gradient-norm mode: ||G||^2 of each tensor (one work-group per tensor), then over the
// table in table order and the scale c = min(1, max_grad_norm / (||G|| + 1e-6)) (NaN
// propagates; one work-group)
__global__ __launch_bounds__(kThreads) void gsum_kernel(const DevTensor *__restrict__ TT, StepConsts k) {
  __shared__ double sh[kThreads];
  const DevTensor &t = TT[blockIdx.x];
  double s = 0.0;
  if (t.n * t.m > 0) {
    if (t.kind != kFactored)
      s = wg_sum(t.ssum, (int64_t)t.ntr * t.ntc * kSub, sh);
    else if (t.zpath)
      s = wg_sum(&t.bst->rsum, t.nzb, sh, sizeof(BandStats) / sizeof(double));
    else
      s = wg_sum(t.rowpart, (int64_t)t.ntc * t.n, sh);
  }
  if (threadIdx.x == 0) stg(k.gsq + blockIdx.x, s);
}
__global__ __launch_bounds__(kThreads) void gnorm_kernel(int ntensors, StepConsts k) {
  __shared__ double sh[kThreads];
  const double total = wg_sum(k.gsq, ntensors, sh);
  if (threadIdx.x == 0) {
    double c = (double)k.max_grad_norm / (sqrt(total) + 1e-6);
    if (c > 1.0) c = 1.0;
    stg(k.gscale, (float)c);
  }
}

// Column factors of the rank-one reconstruction: q = max(mean R, eps) and c'_j = C_j / q
// rounded as the oracle rounds them; b_j = 1/sqrt(c'_j) in double, so that
// 1/D_ij = min(b_j / sqrt(R_i), 1/sqrt(eps)) (Eq. 1 reconstruction with the Alg. 1 clamps).
__device__ __forceinline__ double col_factor(const DevTensor &t, int64_t col, float q) {
  return 1.0 / sqrt((double)(ldg(t.C + col) / q));
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

__device__ __forceinline__ SumPair p2_factored(const DevTensor &t, const Tile &tl, int part, const StepConsts &k,
                                               float q) {
  const WaveMap wm(t, tl);
  const int64_t r0 = wm.wr + (int64_t)part * wm.rpi, rs = (int64_t)wm.rpi * kSub;   // this part's rows
  const int64_t m = t.m, ld = t.ld, col = wm.col;
  const bool mom = t.momentum != 0;
  const float s = mom ? k.s_m : k.s_0;
  const float deps = sqrtf(k.eps);                    // the oracle's D on the floor
  const float reps = (float)(1.0 / (double)deps);     // correctly rounded 1/D
  const float gc = k.gclip ? ldg(k.gscale) : 1.f;     // gradient-norm mode: elements are fl(c g)
  SumPair acc = {0.0, 0.0};
  if (col >= m) return acc;
  float cp[8];    // c'_j = C_j / q, rounded as the oracle
  double bd[8];   // 1/sqrt(c'_j) to about 2^-50 (it scales the unrounded estimate only)
#pragma unroll
  for (int e = 0; e < 8; e++) {
    cp[e] = (col + e < m) ? ldg(t.C + col + e) / q : 0.f;
    const double cd = (double)cp[e];
    bd[e] = (cp[e] > 0.f && cp[e] < __builtin_inff()) ? rsq_d(cd) : 1.0 / sqrt(cd);
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
    for (int64_t lr = r0; lr < tl.nr; lr += 2 * rs) {
      const bool two = lr + rs < tl.nr;
      const int64_t i = tl.row(lr), i2 = two ? tl.row(lr + rs) : i;
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
      if (k.gclip) {
#pragma unroll
        for (int e = 0; e < 8; e++) {
          xa[e] = gc * xa[e];
          xb[e] = gc * xb[e];
        }
      }
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
    for (int64_t lr = r0; lr < tl.nr; lr += rs) {
      const int64_t i = tl.row(lr);
      const float Ri = ldg(t.R + i);
      const double ai = ldg(t.ainv + i);
#pragma unroll
      for (int e = 0; e < 8; e++) {
        if (col + e >= m) continue;
        float x = bf_one(ldg(t.g + i * ld + col + e));
        if (k.gclip) x = gc * x;
        if (mom) x = fmaf(k.a1, x, __fmul_rn(k.b1, ldg(t.M + i * m + col + e)));
        elem(x, Ri, ai, e, acc);
      }
    }
  }
  return acc;
}

// The oracle's own float sequence for U_hat of a factored tensor, summed in double:
// used when the approximate sum leaves the clip factor's rounding undecided.
__device__ __forceinline__ double p2_factored_exact(const DevTensor &t, const Tile &tl, int part,
                                                    const StepConsts &k, float q) {
  const WaveMap wm(t, tl);
  const int64_t r0 = wm.wr + (int64_t)part * wm.rpi, rs = (int64_t)wm.rpi * kSub;
  const int64_t m = t.m, ld = t.ld, col = wm.col;
  const bool mom = t.momentum != 0;
  const float s = mom ? k.s_m : k.s_0;
  const float gc = k.gclip ? ldg(k.gscale) : 1.f;
  double acc = 0.0;
  if (col >= m) return 0.0;
  float cp[8];
#pragma unroll
  for (int e = 0; e < 8; e++) cp[e] = (col + e < m) ? ldg(t.C + col + e) / q : 0.f;
  if (t.vec) {   // 16-byte rows: 8 elements per load
    for (int64_t lr = r0; lr < tl.nr; lr += rs) {
      const int64_t i = tl.row(lr);
      const float Ri = ldg(t.R + i);
      float x[8], mo[8];
      unpack8(ldg(reinterpret_cast<const uint4 *>(t.g + i * ld + col)), x);
      if (mom) load_m8(t.M + i * m + col, mo);
#pragma unroll
      for (int e = 0; e < 8; e++) {
        // the momentum update takes the scaled gradient (as in the update pass)
        const float xs = k.gclip ? gc * x[e] : x[e];
        const float xm = mom ? fmaf(k.a1, xs, __fmul_rn(k.b1, mo[e])) : xs;
        const float u = __fmul_rn(s, xm) / sqrtf(max_nan(__fmul_rn(Ri, cp[e]), k.eps));
        acc = fma((double)u, (double)u, acc);
      }
    }
    return acc;
  }
  for (int64_t lr = r0; lr < tl.nr; lr += rs) {
    const int64_t i = tl.row(lr);
    const float Ri = ldg(t.R + i);
#pragma unroll
    for (int e = 0; e < 8; e++) {
      if (col + e >= m) continue;
      float x = bf_one(ldg(t.g + i * ld + col + e));
      if (k.gclip) x = gc * x;
      if (mom) x = fmaf(k.a1, x, __fmul_rn(k.b1, ldg(t.M + i * m + col + e)));
      const float u = __fmul_rn(s, x) / sqrtf(max_nan(__fmul_rn(Ri, cp[e]), k.eps));
      acc = fma((double)u, (double)u, acc);
    }
  }
  return acc;
}

__device__ __forceinline__ double p2_exact(const DevTensor &t, const Tile &tl, int part, const StepConsts &k) {
  // exact second moment (router tier, vectors): the oracle's operation order exactly
  const WaveMap wm(t, tl);
  const int64_t r0 = wm.wr + (int64_t)part * wm.rpi, rs = (int64_t)wm.rpi * kSub;
  const int64_t m = t.m, ld = t.ld, col = wm.col;
  const bool mom = t.momentum != 0;
  const float gc = k.gclip ? ldg(k.gscale) : 1.f;
  double acc = 0.0;
  for (int64_t lr = r0; lr < tl.nr; lr += rs) {
    const int64_t i = tl.row(lr);
#pragma unroll
    for (int e = 0; e < 8; e++) {
      if (col + e >= m) continue;
      const int64_t sidx = i * m + col + e;
      float g = elem(t.g, i * ld + col + e, t.fp32);
      if (k.gclip) g = gc * g;
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
  const Item it = items[blockIdx.x];   // it.tile = tile * kSub + part
  const DevTensor &t = TT[it.tensor];
  const Tile tl = tile_of(t, it.tile / kSub);
  const int part = it.tile % kSub;
  SumPair acc;
  if (t.kind == kFactored) {
    const float q = mean_r_clamped(t, k, sh);
    acc = p2_factored(t, tl, part, k, q);
  } else {
    acc.s = p2_exact(t, tl, part, k);   // already the oracle's own U_hat
    acc.q4 = 0.0;
  }
  const double s = block_sum(acc.s, sh);
  const double q4 = block_sum(acc.q4, sh);
  if (threadIdx.x == 0) {
    stg(t.ssum + it.tile, s);
    stg(t.qsum + it.tile, q4);
  }
}

// Re-check of the listed tensors over their tiles: level 1 forms the update sum with the
// exact floor test per element (the floored part exactly rounded, the rest unrounded, and
// the sum of U_hat^4 over the rest for its spread); level 2 follows the oracle's float
// sequence exactly. A fixed grid walks the (tensor, tile) pairs of the list.
__device__ __forceinline__ int32_t *recheck_list(RecheckLists *L, int ntensors, int level) {
  int32_t *l1 = reinterpret_cast<int32_t *>(L + 1);
  return level == 1 ? l1 : l1 + ntensors;
}

__global__ __launch_bounds__(kThreads) void recheck_kernel(const DevTensor *__restrict__ TT, RecheckLists *L,
                                                           int ntensors, StepConsts k, int level) {
  __shared__ double sh[kThreads];
  // tile offsets of the listed tensors (an exclusive prefix sum), when the list fits
  constexpr int kTable = 2048;
  __shared__ int64_t pre[kTable + 1];
  __shared__ int64_t part[kThreads];
  const int n = ldg(level == 1 ? &L->n1 : &L->n2);
  if (n <= 0) return;
  const int32_t *list = recheck_list(L, ntensors, level);
  auto tiles = [&](int j) {
    const int32_t ti = ldg(list + j);
    if (ti < 0) return (int64_t)0;   // a slice of a stack whose fast sum is kept
    const DevTensor &t = TT[ti];
    return (int64_t)t.ntr * t.ntc * kSub;   // per-part sums
  };
  const bool table = n <= kTable;
  int64_t total = 0;
  if (table) {
    // thread i sums the counts of entries [8i, 8i + 8), a scan over the threads gives each
    // its start, and it writes its entries' offsets
    constexpr int kPer = kTable / kThreads;
    const int j0 = (int)threadIdx.x * kPer;
    int64_t c[kPer], sum = 0;
#pragma unroll
    for (int q = 0; q < kPer; q++) {
      c[q] = j0 + q < n ? tiles(j0 + q) : 0;
      sum += c[q];
    }
    part[threadIdx.x] = sum;
    __syncthreads();
    for (int off = 1; off < kThreads; off <<= 1) {   // inclusive scan of the thread sums
      const int64_t v = threadIdx.x >= (unsigned)off ? part[threadIdx.x - off] : 0;
      __syncthreads();
      part[threadIdx.x] += v;
      __syncthreads();
    }
    int64_t run = part[threadIdx.x] - sum;
#pragma unroll
    for (int q = 0; q < kPer; q++) {
      pre[j0 + q] = run;
      run += c[q];
    }
    if (threadIdx.x == kThreads - 1) pre[kTable] = run;
    __syncthreads();
    total = pre[n];
  } else {
    for (int j = 0; j < n; j++) total += tiles(j);
  }
  // the tiles of this work-group come in increasing order, so the listed tensor they fall
  // in only moves forward; q is formed once per tensor
  int j = 0, qj = -1;
  int64_t base = 0, nt_j = table ? pre[1] - pre[0] : tiles(0);
  float q = 0.f;
  for (int64_t idx = blockIdx.x; idx < total; idx += gridDim.x) {
    while (idx >= base + nt_j) {
      base += nt_j;
      j++;
      nt_j = table ? pre[j + 1] - pre[j] : tiles(j);
    }
    const DevTensor &t = TT[ldg(list + j)];
    const int tile = (int)(idx - base);   // tile * kSub + part
    const Tile tl = tile_of(t, tile / kSub);
    const int prt = tile % kSub;
    if (j != qj) {
      q = ldg(&t.sc->q);   // the clip stage's q (the one the update pass takes)
      qj = j;
    }
    if (level == 1) {
      const SumPair acc = p2_factored(t, tl, prt, k, q);
      const double sv = block_sum(acc.s, sh);
      const double q4 = block_sum(acc.q4, sh);
      if (threadIdx.x == 0) {
        stg(t.ssum + tile, sv);
        stg(t.qsum + tile, q4);
      }
    } else {
      const double sv = block_sum(p2_factored_exact(t, tl, prt, k, q), sh);
      if (threadIdx.x == 0) stg(t.ssum + tile, sv);
    }
  }
}

// k = 1 / max(1, RMS / d) from the sum S over N elements, rounded once to float (NaN
// propagates); `amb` when a relative spread of S may move k across a rounding boundary of
// the float or across the clipping threshold
__device__ __forceinline__ float clip_from_sum(double S, double N, float d, double spread, bool &amb) {
  const double r = sqrt(S / N) / (double)d;
  const double den = (r != r) ? r : (r < 1.0 ? 1.0 : r);
  const double kd = 1.0 / den;
  const float kf = (float)kd;
  if (!amb && S > 0.0 && r == r && r < 1e300 && spread > 0.0) {
    if (fabs(r - 1.0) <= spread) amb = true;   // at the clipping threshold
    if (r > 1.0) {
      const double up = (double)nextafterf(kf, 3.0e38f), dn = (double)nextafterf(kf, 0.f);
      const double mid_hi = 0.5 * ((double)kf + up), mid_lo = 0.5 * ((double)kf + dn);
      const double tol = 0.5 * spread * kd;
      if (fabs(kd - mid_hi) <= tol || fabs(kd - mid_lo) <= tol) amb = true;
    }
  }
  return kf;
}

// clip factors of the listed tensors from the re-check's sums; level 1 lists for level 2
// the tensors whose spread still leaves k undecided. A stacked tensor's slices are listed
// together; the work-group of its first slice decides k for all of them (one slice per
// wave at a time), the others return.
__global__ __launch_bounds__(kThreads) void clip_recheck_kernel(const DevTensor *__restrict__ TT, RecheckLists *L,
                                                                int ntensors, StepConsts k, int level) {
  __shared__ double sh[kThreads];
  __shared__ double wsum[kWaves][3];
  __shared__ double wek[kWaves];
  __shared__ float kf_sh;
  __shared__ int amb_sh, pos_sh;
  const int n = ldg(level == 1 ? &L->n1 : &L->n2);
  if ((int)blockIdx.x >= n) return;
  const int ti = ldg(recheck_list(L, ntensors, level) + blockIdx.x);
  if (ti < 0) return;
  const DevTensor &t0 = TT[ti];
  if (t0.grp0 != ti) return;
  const int ng = t0.ngrp;
  double S = 0.0, Q4 = 0.0, N = 0.0, Ek = 0.0;   // Ek: error bounds of the kept fast sums
  if (ng == 1) {
    const int64_t ntiles = (int64_t)t0.ntr * t0.ntc * kSub;   // per-part sums
    S = red_sum(RedGroup{sh}, t0.ssum, ntiles);
    if (level == 1) Q4 = red_sum(RedGroup{sh}, t0.qsum, ntiles);
    N = (double)(t0.n * t0.m);
  } else {
    // level 1 re-read only the stack's open slices (and its first); the others, listed as
    // -1 (the group's entries are consecutive from this one), keep the clip stage's fast
    // sum and its error bound
    const int w = (int)(threadIdx.x >> 6);
    double s = 0.0, q4 = 0.0, nn = 0.0, ek = 0.0;
    for (int e = w; e < ng; e += kWaves) {
      const DevTensor &t = TT[ti + e];
      const int64_t ntiles = (int64_t)t.ntr * t.ntc * kSub;
      if (level == 1 && ldg(recheck_list(L, ntensors, 1) + blockIdx.x + e) < 0) {
        s += ldg(&t.sc->s_fast);
        ek += ldg(&t.sc->e_fast);
      } else {
        s += red_sum(RedWave{}, t.ssum, ntiles);
        if (level == 1) q4 += red_sum(RedWave{}, t.qsum, ntiles);
      }
      nn += (double)(t.n * t.m);
    }
    if ((threadIdx.x & 63) == 0) {
      wsum[w][0] = s;
      wsum[w][1] = q4;
      wsum[w][2] = nn;
      wek[w] = ek;
    }
    __syncthreads();
    for (int v = 0; v < kWaves; v++) {   // waves in order
      S += wsum[v][0];
      Q4 += wsum[v][1];
      N += wsum[v][2];
      Ek += wek[v];
    }
  }
  if (threadIdx.x == 0) {
    bool amb = false;
    const double spread = level == 1 ? (20.0 * 0x1p-23 * sqrt(Q4) + Ek) / S + 1e-14 : 0.0;
    if (level == 1) stg(&t0.sc->split_spread, (float)spread);   // for the next step's routing
    kf_sh = clip_from_sum(S, N, k.d, spread, amb);
    amb_sh = amb;
    pos_sh = amb ? atomicAdd(&L->n2, ng) : 0;
  }
  __syncthreads();
  const float kf = kf_sh;
  const bool amb = amb_sh != 0;
  const int pos = pos_sh;
  const int why = ldg(&t0.sc->ambiguous) & ~0xF;
  for (int e = (int)threadIdx.x; e < ng; e += kThreads) {
    if (amb) {
      stg(recheck_list(L, ntensors, 2) + pos + e, (int32_t)(ti + e));
      stg(&TT[ti + e].sc->ambiguous, (int32_t)(kClipPending2 | (kWhySpread << 4)));
    } else {
      stg(&TT[ti + e].sc->k, kf);
      stg(&TT[ti + e].sc->ambiguous, (int32_t)(why | (level == 1 ? kClipSplit : kClipExact)));
    }
  }
}

// One slice's share of the clip stage (a tensor, or one slice of a stacked tensor): the
// estimate of its sum of U_hat^2, the estimate's absolute error bound, and whether its
// floor regime leaves the sum open (the estimate is then an upper bound). Records q and
// the next step's floor regime of the slice.
//
// Row-band tensors: when no element is on the eps floor (min R_i * min c'_j >= eps) the
// sum is sum_j z_j / c'_j, with a spread bounded through max (s x)^2 / (R_i c'_j); when
// every element is (max R_i * max c'_j < eps) it is the exactly rounded floored sum.
// Otherwise both are upper bounds of the oracle's sum (an element's U_hat^2 is at most
// its unfloored and its floored value, up to rounding).
struct SliceSum {
  double S, E;
  int open;     // 0, or why the sum is open (kWhyStraddle, kWhyMissingSum)
  int bad;      // a non-finite sum or statistic
  int repeats;  // the R_i or the c'_j repeat: the spread of the fast sum is not statistical
};

// The spread bounds of the fast sums take the roundings of R_i c'_j, of the square root and
// of the quotient as independent from element to element. When the R_i or the C_j of a
// factored tensor repeat (all equal, as under a constant gradient, or many equal neighbours,
// as under a gradient of a few distinct magnitudes), the first two roundings repeat with
// them and do not average out. Such a tensor takes the rigorous bound instead: each term of
// the fast sum lies within 5.05 u (u = 2^-24) of the oracle's rounded U_hat^2.
constexpr double kRigorousRel = 5.05 * 0x1p-24;
// all (nearly) equal, or more than 1/64 of neighbours equal (never seen with gradients of
// continuous distribution: R_i and C_j are sums of many squares); the extremes are over
// positive values (of R and C, or of R and c' = C / q: the same ratio)
__device__ __forceinline__ int repeats_rule(const DevTensor &t, float rmn, float rmx, float cmn, float cmx,
                                            double dup_r, double dup_c) {
  const bool ur = t.n > 1 && rmx <= rmn * (1.f + 0x1p-20f);
  const bool uc = t.m > 1 && cmx <= cmn * (1.f + 0x1p-20f);
  return (ur || uc || 64.0 * dup_r > (double)t.n || 64.0 * dup_c > (double)t.m) ? 1 : 0;
}
// wide factored tensors: from the fold's per-chunk statistics of R and C (the row-band
// tensors have these in their band and column-chunk statistics)
template <class Red>
__device__ __forceinline__ int repeated_factors(const DevTensor &t, const Red &r) {
  double dup_r = 0.0, dup_c = 0.0;
  float rmn = __builtin_inff(), rmx = 0.f, cmn = __builtin_inff(), cmx = 0.f;
  for (int64_t q = r.lane(); q < (int64_t)t.nfr + t.nfc; q += Red::kN) {
    const ColStats *c = t.cst + q;
    const float mn = ldg(&c->cmin), mx = ldg(&c->cmax);
    const double d = (double)ldg(&c->cdup);
    if (q < t.nfr) {
      rmn = fminf(rmn, mn);
      rmx = fmaxf(rmx, mx);
      dup_r += d;
    } else {
      cmn = fminf(cmn, mn);
      cmx = fmaxf(cmx, mx);
      dup_c += d;
    }
  }
  dup_r = r.sum(dup_r);
  dup_c = r.sum(dup_c);
  rmn = r.minf(rmn);
  rmx = r.maxf(rmx);
  cmn = r.minf(cmn);
  cmx = r.maxf(cmx);
  return repeats_rule(t, rmn, rmx, cmn, cmx, dup_r, dup_c);
}

template <class Red>
__device__ __forceinline__ SliceSum slice_sum(const DevTensor &t, const StepConsts &k, const Red &r) {
  SliceSum o = {0.0, 0.0, 0, 0, 0};
  const float q = t.kind == kFactored ? mean_r_of(t, k, r) : 0.f;
  if (t.kind == kFactored && !t.zpath) o.repeats = repeated_factors(t, r);
  if (t.zpath) {
    const int64_t bstride = sizeof(BandStats) / sizeof(double), cstride = sizeof(ColStats) / sizeof(double);
    const double Y = red_sum(r, &t.bst->ysum, t.nzb, bstride);
    const double SU = red_sum(r, &t.cst->s, t.nfc, cstride);
    // sum over the terms t_ij = (s x)^2 / (R_i c'_j) of t_ij^2 <= umax * sum_j z_j / c'_j^2
    const double SU2 = red_sum(r, &t.cst->s2, t.nfc, cstride);
    double um = 0.0, dup_r = 0.0, dup_c = 0.0;
    float rmn = __builtin_inff(), rmx = 0.f, cmn = __builtin_inff(), cmx = 0.f;
    int bad = 0;
    for (int64_t b = r.lane(); b < t.nzb; b += Red::kN) {
      um = fmax(um, ldg(&t.bst[b].umax));
      rmn = fminf(rmn, ldg(&t.bst[b].rmin));
      rmx = fmaxf(rmx, ldg(&t.bst[b].rmax));
      bad |= ldg(&t.bst[b].bad);
      dup_r += (double)ldg(&t.bst[b].rdup);
    }
    for (int64_t c = r.lane(); c < t.nfc; c += Red::kN) {
      cmn = fminf(cmn, ldg(&t.cst[c].cmin));
      cmx = fmaxf(cmx, ldg(&t.cst[c].cmax));
      bad |= ldg(&t.cst[c].bad);
      dup_c += (double)ldg(&t.cst[c].cdup);
    }
    um = r.max(um);
    rmn = r.minf(rmn);
    rmx = r.maxf(rmx);
    cmn = r.minf(cmn);
    cmx = r.maxf(cmx);
    bad = r.any(bad);
    o.repeats = repeats_rule(t, rmn, rmx, cmn, cmx, r.sum(dup_r), r.sum(dup_c));
    // the sums the row-band pass formed this step (it skips one when the last step
    // predicts the regime); a sum it did not form counts as +inf
    const int formed = ldg(&t.bst[0].regime);
    const bool have_z = formed != kRegimeFloor, have_y = formed != kRegimeAbove;
    const double inf = __builtin_inf();
    const double SUf = have_z ? SU : inf, Yf = have_y ? Y : inf;
    const bool finite = !(SUf != SUf) && !(Yf != Yf) && (SUf < 1e300 || Yf < 1e300);
    const float lo = __fmul_rn(rmn, cmn), hi = __fmul_rn(rmx, cmx);
    if (bad || !finite) {
      o.bad = 1;
      o.S = SU;
    } else if (have_z && lo >= k.eps) {   // nothing on the floor
      o.S = SU;
      o.E = SU > 0.0 ? 20.0 * 0x1p-23 * sqrt(um * SU2) + 1e-14 * SU : 0.0;
      if (o.repeats) o.E = fmax(o.E, kRigorousRel * SU + 1e-14 * SU);
    } else if (have_y && hi < k.eps) {    // everything on the floor
      o.S = Y;
      o.E = 1e-14 * Y;
    } else {
      o.S = fmin(SUf, Yf) * (1.0 + 1e-6);  // an upper bound of the oracle's sum
      o.open = (have_z && have_y) ? kWhyStraddle : kWhyMissingSum;
    }
    // the next step's prediction. Without new gradient R_i c'_j only decays by beta2 per
    // step, but a larger gradient can lift it by any factor: a 5% margin above the floor,
    // a factor 2 below it. A wrong prediction costs a re-check at most.
    const int next = (lo >= 1.05f * k.eps) ? kRegimeAbove : (2.f * hi < k.eps ? kRegimeFloor : kRegimeBoth);
    if (r.lead()) stg(&t.sc->regime, o.bad ? (int32_t)kRegimeBoth : (int32_t)next);
  } else {
    const int64_t ntiles = (int64_t)t.ntr * t.ntc * kSub;   // per-part sums
    o.S = red_sum(r, t.ssum, ntiles);
    const double Q4 = red_sum(r, t.qsum, ntiles);
    // the exact second moment's sum is the oracle's own; a factored one carries the
    // spread of its unrounded terms (20 standard deviations)
    o.E = t.kind == kFactored ? 20.0 * 0x1p-23 * sqrt(Q4) + 1e-14 * o.S : 0.0;
    if (o.repeats) o.E = fmax(o.E, kRigorousRel * o.S + 1e-14 * o.S);
  }
  if (r.lead()) stg(&t.sc->q, q);
  return o;
}

// The clip stage's share of each slice of the stacked tensors, one wave per slice: its fast
// sum, error bound and flags (kept in its scalars for the group's decision and, should the
// stack's sum be open, for its re-check), its q and its next regime.
__global__ __launch_bounds__(kThreads) void clip_slices_kernel(const DevTensor *__restrict__ TT,
                                                               const Item *__restrict__ items, int64_t count,
                                                               StepConsts k) {
  const int64_t j = (int64_t)blockIdx.x * kWaves + (threadIdx.x >> 6);
  if (j >= count) return;   // a whole wave
  const DevTensor &t = TT[items[j].tensor];
  const SliceSum o = slice_sum(t, k, RedWave{});
  if ((threadIdx.x & 63) == 0) {
    stg(&t.sc->s_fast, o.S);
    stg(&t.sc->e_fast, o.E);
    stg(&t.sc->fast_flags, (int32_t)((o.open & 15) | (o.bad ? 16 : 0) | (o.repeats ? 32 : 0)));
  }
}

// --------------------------------------------------------------------------------------------
// clip stage, one work-group per tensor (or per stacked tensor, whose slices share one k):
// k = 1 / max(1, RMS(U_hat) / d) (Sec. 3, Alg. 1), NaN-propagating and rounded once to
// float as the oracle rounds it. It records q = max(mean R, eps) and flags the tensor when
// k's rounding is not decided by the approximate sum: its spread (20 standard deviations
// of the free roundings) reaches a rounding boundary of k or the clipping threshold. When
// a slice's floor regime leaves its sum open, the group's sum is an upper bound: below
// the clipping threshold k is exactly 1, and above it the tensor goes to a re-check.
// --------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kThreads) void clip_kernel(const DevTensor *__restrict__ TT,
                                                        const Item *__restrict__ items, StepConsts k,
                                                        RecheckLists *L, int ntensors) {
  __shared__ double sh[kThreads];
  __shared__ double wsum[kWaves][3];
  __shared__ int wflag[kWaves][4];
  __shared__ float kf_sh;
  __shared__ int st_sh, pos_sh;
  // a stack's open slices, for a floor-split re-check of those alone (stacks of up to
  // kOpenBits slices; a larger one re-reads every slice)
  constexpr int kOpenBits = 32 * 64;
  __shared__ uint32_t openbits[kOpenBits / 32];
  const Item it = items[blockIdx.x];   // the first sub-tensor of a group sharing one k
  const DevTensor &t0 = TT[it.tensor];
  const int g0 = t0.grp0, ng = t0.ngrp;
  // the group's sum S as the sum of its slices' estimates, with the sum of their absolute
  // error bounds, in slice order within a wave and then wave by wave
  double S = 0.0, err = 0.0, N = 0.0;
  int open = 0;   // why the first open slice (in slice order) is open
  bool bad_any = false, rep_any = false;
  if (ng == 1) {
    const SliceSum o = slice_sum(t0, k, RedGroup{sh});
    S = o.S;
    err = o.E;
    N = (double)(t0.n * t0.m);
    open = o.open;
    bad_any = o.bad != 0;
    rep_any = o.repeats != 0;
  } else {
    // the slices' sums come from clip_slices_kernel (launched just before)
    for (int q = (int)threadIdx.x; q < kOpenBits / 32; q += kThreads) openbits[q] = 0u;
    __syncthreads();
    const int w = (int)(threadIdx.x >> 6);
    double s = 0.0, e_ = 0.0, nn = 0.0;
    int first = 0x7fffffff, why = 0, bad = 0, rep = 0;   // the wave's first open slice, and why it is open
    for (int e = w; e < ng; e += kWaves) {
      const DevTensor &t = TT[g0 + e];
      const int fl = ldg(&t.sc->fast_flags);
      const SliceSum o = {ldg(&t.sc->s_fast), ldg(&t.sc->e_fast), fl & 15, (fl >> 4) & 1, (fl >> 5) & 1};
      if ((threadIdx.x & 63) == 0 && o.open && e < kOpenBits) atomicOr(&openbits[e >> 5], 1u << (e & 31));
      s += o.S;
      e_ += o.E;
      nn += (double)(t.n * t.m);
      if (o.open && first == 0x7fffffff) {
        first = e;
        why = o.open;
      }
      bad |= o.bad;
      rep |= o.repeats;
    }
    if ((threadIdx.x & 63) == 0) {
      wsum[w][0] = s;
      wsum[w][1] = e_;
      wsum[w][2] = nn;
      wflag[w][0] = first;
      wflag[w][1] = why;
      wflag[w][2] = bad;
      wflag[w][3] = rep;
    }
    __syncthreads();
    int f = 0x7fffffff;
    for (int v = 0; v < kWaves; v++) {   // waves in order
      S += wsum[v][0];
      err += wsum[v][1];
      N += wsum[v][2];
      if (wflag[v][0] < f) {
        f = wflag[v][0];
        open = wflag[v][1];
      }
      bad_any |= wflag[v][2] != 0;
      rep_any |= wflag[v][3] != 0;
    }
  }
  if (threadIdx.x == 0) {
    bool amb = (k.flags & SKEW_FLAG_EXACT_CLIP) != 0 && t0.kind == kFactored;
    int why = amb ? kWhyForced : (open ? open : 0);
    int level = 2;   // the re-check a flagged group gets
    double spread = 0.0;
    if (bad_any) {
      amb = true;
      why = kWhyNonFinite;
    } else if (open) {
      S += err;   // an upper bound of the group's sum
      if (!(sqrt(S / N) / (double)k.d < 1.0) && !amb) {
        amb = true;
        // the floor split per element decides most of these, except where the factors
        // repeat (its spread is statistical too). A tensor whose terms left the split's
        // spread wide (heavy tails) keeps them from step to step: when the last split's
        // relative spread makes an undecided k likely (more than 0.55 of the spacing of k's
        // floats near the estimate: the exact sequence costs about 1/0.45 of the split's
        // vector work), it goes straight to the exact sequence. Every eighth step takes
        // the split, which renews the spread. The choice only saves a pass.
        const double r = sqrt(S / N) / (double)k.d;
        const float kg = (float)(1.0 / r);
        const double gap = (double)nextafterf(kg, 3.0e38f) - (double)kg;
        const bool wide = (double)ldg(&t0.sc->split_spread) * (1.0 / r) > 0.55 * gap && (k.step & 7) != 0;
        level = (rep_any || wide) ? 2 : 1;
      }
    } else {
      spread = S > 0.0 ? err / S : 0.0;
    }
    const bool flagged_before = amb;
    kf_sh = clip_from_sum(S, N, k.d, spread, amb);
    if (amb && !flagged_before) why = kWhySpread;
    const bool list = amb && t0.kind == kFactored;
    pos_sh = list ? atomicAdd(level == 1 ? &L->n1 : &L->n2, ng) : 0;
    st_sh = list ? (int)((level == 1 ? kClipPending1 : kClipPending2) | (why << 4)) | (level << 16) : -1;
  }
  __syncthreads();
  const float kf = kf_sh;
  const int st = st_sh, pos = pos_sh;
  // a stack's floor-split re-check reads its first slice (whose work-group decides k) and
  // its open slices; the others are listed as -1 and keep their fast sums
  const bool partial = (st >> 16) == 1 && ng > 1 && ng <= kOpenBits;
  for (int e = (int)threadIdx.x; e < ng; e += kThreads) {
    const DevTensor &t = TT[g0 + e];
    stg(&t.sc->k, kf);
    if (st >= 0) {
      const bool keep = partial && e > 0 && !((openbits[e >> 5] >> (e & 31)) & 1u);
      stg(recheck_list(L, ntensors, st >> 16) + pos + e, keep ? (int32_t)-1 : (int32_t)(g0 + e));
      stg(&t.sc->ambiguous, (int32_t)(st & 0xFFFF));
    } else {
      stg(&t.sc->ambiguous, (int32_t)kClipFast);
    }
  }
}

// The weight the update starts from: w - (lr lambda) w with one rounding when the decoupled
// weight decay applies (Sec. 3 footnote, Sec. 6), else w itself
__device__ __forceinline__ float decayed(float w, bool dec, float wd) { return dec ? fmaf(-wd, w, w) : w; }

// The oracle's float sequence for one factored element (Alg. 1 with the eps clamps):
// D = sqrt(max(R_i * c'_j, eps)), U = ((s * x) / D) * k, y = (wd - lr U) + xi, where wd is
// the (decayed) starting weight and xi scales with the pre-step |w|.
__device__ __forceinline__ float exact_factored_y(float x, float w, float wd, float Ri, float cpj, float s,
                                                  float kc, float eps, float lr, float dith, bool xu) {
  const float vh = __fmul_rn(Ri, cpj);
  const float dd = sqrtf(max_nan(vh, eps));
  const float U = __fmul_rn(__fmul_rn(s, x) / dd, kc);
  return fmaf(dith, dither_mul(w, xu), fmaf(-lr, U, wd));
}

// y may round differently from the oracle's value when this is >= 0: the fast update x*F
// differs from the oracle's lr*U by < 2^-19 relative, and each of x and y carries one
// rounding. (y - mid is exact and finite for finite y; NaN never counts as near.)
__device__ __forceinline__ float boundary_slack(float y, float xF, float w) {
  // the midpoint between y's two bf16 neighbours: y's high half, then 0x8000
  const float mid = __uint_as_float(__builtin_amdgcn_perm(__float_as_uint(y), 0x8000u, 0x07060100u));
  const float bound = fmaf(fabsf(xF), 0x1p-18f + 0x1p-21f, fabsf(w) * 0x1p-21f);
  return bound - fabsf(y - mid);
}
__device__ __forceinline__ bool near_boundary(float y, float xF, float w) { return boundary_slack(y, xF, w) >= 0.f; }

struct P3Scalars {
  float q, s, kc, cap3, eps, lr, gc;
  double lsk;
};

// one row segment of 8 elements (vector path): momentum, update, dither, bf16 store.
// The fast path forms 1/D from per-row and per-column factors; the few elements whose
// result might round to the other bf16 neighbour take the oracle's exact sequence.
template <bool XU, bool DEC, bool GC>
__device__ __forceinline__ void p3_row8(const DevTensor &t, const StepConsts &k, const P3Scalars &c,
                                        const Dither &dz, int64_t i, int64_t col, const float *bf, uint4 gw,
                                        uint4 ww, const float *mv) {
  const bool mom = t.momentum != 0;
  float x[8], w[8];
  unpack8(gw, x);
  unpack8(ww, w);
  if (GC) {
#pragma unroll
    for (int e = 0; e < 8; e++) x[e] = c.gc * x[e];
  }
  if (mom) {
#pragma unroll
    for (int e = 0; e < 8; e++) x[e] = fmaf(k.a1, x[e], __fmul_rn(k.b1, mv[e]));
    store_m8(t.M + i * t.m + col, x);
  }
  const float alpha = (float)(c.lsk * ldg(t.ainv + i));
  // pairs p0 .. p0 + 3: m and col are multiples of 8, so p0 is a multiple of 4 and the
  // four pairs share their high word and differ only in the low two bits
  const uint64_t p0 = ((uint64_t)t.idx0 + (uint64_t)i * (uint64_t)t.m + (uint64_t)col) >> 1;
  // pair indices reach 2^32 only in tensors of more than 2^33 elements (a uniform test)
  const uint32_t base =
      (t.idx0 + t.n * t.m > (int64_t(1) << 33)) ? dz.pair_base(p0) : ((uint32_t)p0 ^ dz.klo ^ dz.inner0);
  float y[8], dith[8];
#pragma unroll
  for (int e2 = 0; e2 < 4; e2++) {
    const uint32_t h = fmix32(base ^ (uint32_t)e2);
    dith[2 * e2] = dither_lo(h);
    dith[2 * e2 + 1] = dither_hi(h);
  }
  const bool dec = DEC && t.decay;
  constexpr bool xu = XU;
  float slack = -1.f;
#pragma unroll
  for (int e = 0; e < 8; e++) {
    const float F = fminf(alpha * bf[e], c.cap3);
    y[e] = fmaf(dith[e], dither_mul(w[e], xu), fmaf(-x[e], F, decayed(w[e], dec, k.wd)));
    slack = fmaxf(slack, boundary_slack(y[e], x[e] * F, w[e]));
  }
  if (slack >= 0.f) {
    const float Ri = ldg(t.R + i);
#pragma unroll
    for (int e = 0; e < 8; e++) {
      const float F = fminf(alpha * bf[e], c.cap3);
      if (near_boundary(y[e], x[e] * F, w[e]))
        y[e] = exact_factored_y(x[e], w[e], decayed(w[e], dec, k.wd), Ri, ldg(t.C + col + e) / c.q, c.s, c.kc,
                                c.eps, c.lr, dith[e], xu);
    }
  }
  stg_nt(reinterpret_cast<uint4 *>(t.w + i * t.ld + col),
         make_uint4(pack_bf16x2(y[0], y[1]), pack_bf16x2(y[2], y[3]), pack_bf16x2(y[4], y[5]),
                    pack_bf16x2(y[6], y[7])));
}

template <bool XU, bool DEC, bool GC>
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
  c.gc = GC ? ldg(k.gscale) : 1.f;             // gradient-norm mode: elements are fl(c g)
  c.cap3 = (float)(c.lsk / (double)sqrtf(k.eps));
  if (t.vec) {
    float bf[8];
#pragma unroll
    for (int e = 0; e < 8; e++) bf[e] = (float)col_factor(t, col + e, c.q);
    for (int64_t lr = wm.wr; lr < tl.nr; lr += 2 * wm.rpi) {
      const bool two = lr + wm.rpi < tl.nr;
      const int64_t i = tl.row(lr), i2 = two ? tl.row(lr + wm.rpi) : i;
      const uint4 ga = ldg_nt(reinterpret_cast<const uint4 *>(t.g + i * ld + col));
      const uint4 wa = ldg_nt(reinterpret_cast<const uint4 *>(t.w + i * ld + col));
      const uint4 gb = ldg_nt(reinterpret_cast<const uint4 *>(t.g + i2 * ld + col));
      const uint4 wb = ldg_nt(reinterpret_cast<const uint4 *>(t.w + i2 * ld + col));
      float ma[8], mb[8];
      if (mom) {
        load_m8(t.M + i * m + col, ma);
        load_m8(t.M + i2 * m + col, mb);
      }
      p3_row8<XU, DEC, GC>(t, k, c, dz, i, col, bf, ga, wa, ma);
      if (two) p3_row8<XU, DEC, GC>(t, k, c, dz, i2, col, bf, gb, wb, mb);
    }
  } else {
    for (int64_t lr = wm.wr; lr < tl.nr; lr += wm.rpi) {
    const int64_t i = tl.row(lr);
      const float alpha = (float)(c.lsk * ldg(t.ainv + i));
      const uint64_t rowidx = (uint64_t)t.idx0 + (uint64_t)i * (uint64_t)m;
#pragma unroll
      for (int e = 0; e < 8; e++) {
        if (col + e >= m) continue;
        float x = bf_one(ldg(t.g + i * ld + col + e));
        const float w = bf_one(ldg(t.w + i * ld + col + e));
        if (GC) x = c.gc * x;
        if (mom) {
          x = fmaf(k.a1, x, __fmul_rn(k.b1, ldg(t.M + i * m + col + e)));
          stg(t.M + i * m + col + e, x);
        }
        const uint64_t idx = rowidx + (uint64_t)(col + e);
        const float dith = dither_of(dz.pair(idx >> 1), idx);
        const float F = fminf(alpha * (float)col_factor(t, col + e, c.q), c.cap3);
        const float wd = decayed(w, DEC && t.decay, k.wd);
        constexpr bool xu = XU;
        float y = fmaf(dith, dither_mul(w, xu), fmaf(-x, F, wd));
        if (near_boundary(y, x * F, w))
          y = exact_factored_y(x, w, wd, ldg(t.R + i), ldg(t.C + col + e) / c.q, c.s, kc, k.eps, k.lr, dith, xu);
        stg(t.w + i * ld + col + e, to_bf16(y));
      }
    }
  }
}

template <bool XU, bool DEC, bool GC>
__device__ __forceinline__ void p3_exact(const DevTensor &t, const Tile &tl, const StepConsts &k, float kc,
                                         const Dither &dz) {
  // exact second moment: the oracle's operation order exactly
  const WaveMap wm(t, tl);
  const int64_t m = t.m, ld = t.ld, col = wm.col;
  const bool mom = t.momentum != 0;
  const float gc = GC ? ldg(k.gscale) : 1.f;
  for (int64_t lr = wm.wr; lr < tl.nr; lr += wm.rpi) {
    const int64_t i = tl.row(lr);
#pragma unroll
    for (int e = 0; e < 8; e++) {
      if (col + e >= m) continue;
      const int64_t sidx = i * m + col + e;
      float g = elem(t.g, i * ld + col + e, t.fp32);
      if (GC) g = gc * g;
      const float w = elem(t.w, i * ld + col + e, t.fp32);
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
      const float x = fmaf(-k.lr, U, decayed(w, DEC && t.decay, k.wd));
      if (t.fp32) {   // float32 master: no dither, no cast
        stg(reinterpret_cast<float *>(t.w) + i * ld + col + e, x);
        continue;
      }
      const uint64_t idx = (uint64_t)(t.idx0 + sidx);
      constexpr bool xu = XU;
      const float y = fmaf(dither_of(dz.pair(idx >> 1), idx), dither_mul(w, xu), x);
      stg(t.w + i * ld + col + e, to_bf16(y));
    }
  }
}

// --------------------------------------------------------------------------------------------
// p3: clip factor, state update, weight update and dithered bf16 write-back (Alg. 1)
// --------------------------------------------------------------------------------------------
// XU: the exact-ulp dither; DEC: the decoupled weight decay is on (lr lambda != 0); GC: the
// gradient-norm mode (elements enter as fl(c g))
// (at most 128 VGPRs: four waves per SIMD keep enough loads in flight)
template <bool XU, bool DEC, bool GC>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4))) void p3_kernel(const DevTensor *__restrict__ TT,
                                                      const Item *__restrict__ items, StepConsts k,
                                                      RecheckLists *L) {
  // the re-check lists of this step are consumed: empty them for the next
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    stg(&L->n1, 0);
    stg(&L->n2, 0);
  }
  const Item it = items[blockIdx.x];
  const DevTensor &t = TT[it.tensor];
  const Tile tl = tile_of(t, it.tile);
  const float kc = ldg(&t.sc->k);
  const Dither dz(k.seed, k.step, t.tensor_id);
  if (t.kind == kFactored)
    p3_factored<XU, DEC, GC>(t, tl, k, kc, ldg(&t.sc->q), dz);
  else
    p3_exact<XU, DEC, GC>(t, tl, k, kc, dz);
}

}  // namespace

// The static workspace of skew_state_init_static: device memory the library itself holds
// on every GPU it runs on, for callers that cannot allocate. Host code never passes the
// array's name to a kernel or a copy: it takes the array's device address on each device
// from hipGetSymbolAddress (looked up once per device, with that device current).
static __device__ __align__(256) unsigned char scratch[SKEW_STATIC_WORKSPACE_BYTES];

int static_workspace(void **ptr) {
  constexpr int kMaxDev = 64;
  static std::mutex mu;
  static void *addr[kMaxDev] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return (int)e;
  if (dev < 0 || dev >= kMaxDev) return (int)hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(mu);
  if (addr[dev] == nullptr) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return (int)e;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return (int)hipSuccess;
}

int launch_p1(const DevTensor *T, const Item *items, int64_t count, void *stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(p1_kernel, dim3((uint32_t)count), dim3(kThreads), 0, (hipStream_t)stream, T, items);
  return (int)hipGetLastError();
}
int launch_p1z(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, int variant, int mode,
               void *stream) {
  if (count <= 0) return hipSuccess;
  const dim3 grid((uint32_t)count), block(kZThreads);
  hipStream_t s = (hipStream_t)stream;
  switch (variant) {
#define SKEW_P1Z_CASE(V, NSEG, VEC, MOM)                                                          \
  case V:                                                                                          \
    if (mode == 1)                                                                                 \
      hipLaunchKernelGGL((p1z_kernel<NSEG, MOM, VEC, true, (NSEG <= 2 && VEC && !MOM) ? 1 : 0>), grid, \
                         block, 0, s, T, items, k, 1);                                            \
    else if (mode == 2)                                                                            \
      hipLaunchKernelGGL((p1z_kernel<NSEG, MOM, VEC, true, (NSEG <= 2 && VEC && !MOM) ? 2 : 0>), grid, \
                         block, 0, s, T, items, k, 2);                                            \
    else if (mode != 0)                                                                            \
      hipLaunchKernelGGL((p1z_kernel<NSEG, MOM, VEC, true>), grid, block, 0, s, T, items, k, mode); \
    else                                                                                           \
      hipLaunchKernelGGL((p1z_kernel<NSEG, MOM, VEC, false>), grid, block, 0, s, T, items, k, 0);  \
    break;
    SKEW_P1Z_CASE(0, 1, true, false)
    SKEW_P1Z_CASE(1, 1, true, true)
    SKEW_P1Z_CASE(2, 1, false, false)
    SKEW_P1Z_CASE(3, 1, false, true)
    SKEW_P1Z_CASE(4, 2, true, false)
    SKEW_P1Z_CASE(5, 2, true, true)
    SKEW_P1Z_CASE(6, 2, false, false)
    SKEW_P1Z_CASE(7, 2, false, true)
    SKEW_P1Z_CASE(8, 4, true, false)
    SKEW_P1Z_CASE(9, 4, true, true)
    SKEW_P1Z_CASE(10, 4, false, false)
    SKEW_P1Z_CASE(11, 4, false, true)
    SKEW_P1Z_CASE(12, 3, true, false)
    SKEW_P1Z_CASE(14, 3, false, false)
#undef SKEW_P1Z_CASE
    default: return (int)hipErrorInvalidValue;
  }
  return (int)hipGetLastError();
}
int launch_fold(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, int phase, void *stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(fold_kernel, dim3((uint32_t)count), dim3(kThreads), 0, (hipStream_t)stream, T, items, k, phase);
  return (int)hipGetLastError();
}
int launch_gsq(const DevTensor *T, const Item *items, int64_t count, void *stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(gsq_kernel, dim3((uint32_t)count), dim3(kThreads), 0, (hipStream_t)stream, T, items);
  return (int)hipGetLastError();
}
int launch_gnorm(const DevTensor *T, int ntensors, const StepConsts &k, void *stream) {
  if (ntensors <= 0) return hipSuccess;
  hipLaunchKernelGGL(gsum_kernel, dim3((uint32_t)ntensors), dim3(kThreads), 0, (hipStream_t)stream, T, k);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return (int)e;
  hipLaunchKernelGGL(gnorm_kernel, dim3(1), dim3(kThreads), 0, (hipStream_t)stream, ntensors, k);
  return (int)hipGetLastError();
}
int launch_p2(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, void *stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(p2_kernel, dim3((uint32_t)count), dim3(kThreads), 0, (hipStream_t)stream, T, items, k);
  return (int)hipGetLastError();
}
int launch_clip_slices(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, void *stream) {
  if (count <= 0) return hipSuccess;
  const int64_t groups = (count + kWaves - 1) / kWaves;
  hipLaunchKernelGGL(clip_slices_kernel, dim3((uint32_t)groups), dim3(kThreads), 0, (hipStream_t)stream, T, items,
                     count, k);
  return (int)hipGetLastError();
}
int launch_clip(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, RecheckLists *L,
                int ntensors, void *stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL(clip_kernel, dim3((uint32_t)count), dim3(kThreads), 0, (hipStream_t)stream, T, items, k, L,
                     ntensors);
  return (int)hipGetLastError();
}
int launch_recheck(const DevTensor *T, RecheckLists *L, int ntensors, const StepConsts &k, int level, void *stream) {
  if (ntensors <= 0) return hipSuccess;
  hipLaunchKernelGGL(recheck_kernel, dim3(kRecheckGrid), dim3(kThreads), 0, (hipStream_t)stream, T, L, ntensors, k,
                     level);
  return (int)hipGetLastError();
}
int launch_clip_recheck(const DevTensor *T, RecheckLists *L, int ntensors, const StepConsts &k, int level,
                        void *stream) {
  if (ntensors <= 0) return hipSuccess;
  hipLaunchKernelGGL(clip_recheck_kernel, dim3((uint32_t)ntensors), dim3(kThreads), 0, (hipStream_t)stream, T, L,
                     ntensors, k, level);
  return (int)hipGetLastError();
}
int launch_p3(const DevTensor *T, const Item *items, int64_t count, const StepConsts &k, RecheckLists *L,
              void *stream) {
  if (count <= 0) return hipSuccess;
  const bool xu = (k.flags & SKEW_FLAG_EXACT_ULP) != 0, dec = k.wd != 0.f, gc = k.gclip != 0;
  auto *kern = xu ? (dec ? (gc ? p3_kernel<true, true, true> : p3_kernel<true, true, false>)
                         : (gc ? p3_kernel<true, false, true> : p3_kernel<true, false, false>))
                  : (dec ? (gc ? p3_kernel<false, true, true> : p3_kernel<false, true, false>)
                         : (gc ? p3_kernel<false, false, true> : p3_kernel<false, false, false>));
  hipLaunchKernelGGL(kern, dim3((uint32_t)count), dim3(kThreads), 0, (hipStream_t)stream, T, items, k, L);
  return (int)hipGetLastError();
}

}  // namespace skew
