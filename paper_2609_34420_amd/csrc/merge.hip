// LSE merge of context-parallel partials (Section III-A-1 part 3):
//   LSE = log sum_p exp(LSE_p),  O = sum_p exp(LSE_p - LSE) O_p.
// HBM-bound elementwise pass: one thread per (row, 4 features), float4 loads.
#include "common.hpp"
#include "kernels.hpp"

namespace gt {

namespace {

template <bool OUT_BF16>
__global__ __launch_bounds__(256) void merge_kernel(MergeArgs a) {
  const int cpr = a.d >> 2;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = idx / cpr;
  const int ch = (int)(idx % cpr);
  if (row >= a.rows) return;
  float m = -INFINITY;
  for (int p = 0; p < a.n_parts; ++p) m = fmaxf(m, a.lse_parts[(int64_t)p * a.rows + row]);
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  float lse = -INFINITY;
  if (m != -INFINITY) {
    float tot = 0.0f;
    for (int p = 0; p < a.n_parts; ++p) tot += expf(a.lse_parts[(int64_t)p * a.rows + row] - m);
    const float inv = 1.0f / tot;
    for (int p = 0; p < a.n_parts; ++p) {
      const float w = expf(a.lse_parts[(int64_t)p * a.rows + row] - m) * inv;
      if (w == 0.0f) continue;
      const float4 v = *reinterpret_cast<const float4*>(a.o_parts + ((int64_t)p * a.rows + row) * a.d + ch * 4);
      acc.x = fmaf(w, v.x, acc.x);
      acc.y = fmaf(w, v.y, acc.y);
      acc.z = fmaf(w, v.z, acc.z);
      acc.w = fmaf(w, v.w, acc.w);
    }
    lse = m + logf(tot);
  }
  if constexpr (OUT_BF16) {
    uint2 pk;
    pk.x = (uint32_t)f2bf(acc.x) | ((uint32_t)f2bf(acc.y) << 16);
    pk.y = (uint32_t)f2bf(acc.z) | ((uint32_t)f2bf(acc.w) << 16);
    *reinterpret_cast<uint2*>(reinterpret_cast<uint16_t*>(a.o) + row * a.d + ch * 4) = pk;
  } else {
    *reinterpret_cast<float4*>(reinterpret_cast<float*>(a.o) + row * a.d + ch * 4) = acc;
  }
  if (ch == 0) a.lse[row] = lse;
}

}  // namespace

hipError_t launch_merge(const MergeArgs& a, bool out_bf16, hipStream_t s) {
  const int64_t threads = a.rows * (a.d / 4);
  const unsigned grid = (unsigned)((threads + 255) / 256);
  if (out_bf16)
    hipLaunchKernelGGL(merge_kernel<true>, dim3(grid), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(merge_kernel<false>, dim3(grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace gt
