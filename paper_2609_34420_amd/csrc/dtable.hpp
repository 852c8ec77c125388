// Bias-table gradient, dtable[h, b] = sum of dS[i, j] over the pairs with
// spd[i, j] = b, accumulated in a fixed-point LDS histogram (the vector-ALU
// dQ kernel; the matrix-core dK/dV kernel keeps its own copy of these steps
// inline, where the shared form cost it 2.5 % through register allocation).
//
// LDS float atomics are slow on this hardware and 64-bit integer adds are
// not, so dS is accumulated as round(dS 2^F) in 64-bit integers. The power of
// two per head keeps every term below 2^30 in magnitude:
//   |dS_ij| <= |dO_i . V_j - Dlt_i| <= max_i |dO_i| max_j |V_j| + max_i |Dlt_i|
// (P_ij <= 1, Cauchy-Schwarz), and the prepare stage records block maxima of
// |dO_i|^2, |V_j|^2 and |Dlt_i|. Dlt enters on its own because in a ring step
// O mixes the values of every key block, not only of the keys at hand. Sums
// of up to 2^32 terms fit in 64 bits. Each workgroup flushes its histogram
// once, converted back to fp32, with one global atomic per bucket.
#pragma once
#include "common.hpp"
#include "kernels.hpp"

namespace gt {

__device__ __forceinline__ int round_to_int(float x) {
  int r;
  asm("v_cvt_rpi_i32_f32 %0, %1" : "=v"(r) : "v"(x));   // floor(x + 0.5)
  return r;
}

// Fixed-point exponent F of head h: (max|dO| max|V| + max|Dlt|) 2^F <= 2^30
// (a 1.5 % margin covers the rounding of P and of the products). Every
// thread of the workgroup calls it; red is NW x 3 floats of LDS. Contains a
// workgroup barrier.
template <int NW>
__device__ __forceinline__ int hist_exponent(const BwdArgs& a, int h, float (*red)[NW]) {
  const int tid = threadIdx.x;
  const int wave = wave_id();
  {
    const int64_t nblk = ((a.Sq > a.Sk ? a.Sq : a.Sk) + 255) / 256;
    const float* nm = a.nmax + (int64_t)h * nblk * 4;
    float md = 0.0f, mv = 0.0f, ml = 0.0f;
    for (int64_t t = tid; t < nblk; t += NW * 64) {
      md = fmaxf(md, nm[4 * t]);
      mv = fmaxf(mv, nm[4 * t + 1]);
      ml = fmaxf(ml, nm[4 * t + 2]);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      md = fmaxf(md, __shfl_xor(md, off));
      mv = fmaxf(mv, __shfl_xor(mv, off));
      ml = fmaxf(ml, __shfl_xor(ml, off));
    }
    if ((tid & 63) == 0) {
      red[0][wave] = md;
      red[1][wave] = mv;
      red[2][wave] = ml;
    }
  }
  __syncthreads();
  float md = red[0][0], mv = red[1][0], ml = red[2][0];
#pragma unroll
  for (int w = 1; w < NW; ++w) {
    md = fmaxf(md, red[0][w]);
    mv = fmaxf(mv, red[1][w]);
    ml = fmaxf(ml, red[2][w]);
  }
  const float bound = 1.015f * (sqrtf(md) * sqrtf(mv) + ml);
  int fexp = 40;
  if (bound > 0.0f && bound < INFINITY) {
    int e;
    frexpf(bound, &e);                 // bound < 2^e
    fexp = 30 - e;
    fexp = fexp > 40 ? 40 : (fexp < -100 ? -100 : fexp);
  }
  return fexp;
}

// Adds the workgroup's histogram (entry (b, c) at hist[b * CPY + c]) to
// dtable_h[0 .. n_buckets). Call after a barrier that follows the last add.
template <int CPY>
__device__ __forceinline__ void flush_hist(const unsigned long long* hist, int n_buckets, int fexp, float* dtable_h,
                           int nthreads) {
  const double unscale = ldexp(1.0, -fexp);
  for (int bkt = threadIdx.x; bkt < n_buckets; bkt += nthreads) {
    long long t = 0;
#pragma unroll
    for (int c = 0; c < CPY; ++c) t += (long long)hist[bkt * CPY + ((c + bkt) & (CPY - 1))];
    if (t != 0) atomicAdd(&dtable_h[bkt], (float)((double)t * unscale));
  }
}

}  // namespace gt
