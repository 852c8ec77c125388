// Forward / ring-step kernels: blockwise biased attention with online softmax.
//
// S = scale * Q K^T + table[h, spd[row_off + i, col_off + j]]   (Eq. (1); Eq. (2)
// for a ring step), softmax statistics updated block by block with the bias
// already inside the scores (Section III-A-1 part 3).
//
// bf16 path (gfx950 matrix cores). Each wave owns 32*QB queries and computes
// the TRANSPOSED score tile S^T = K Q^T, so every lane owns one query
// (lane & 31) and 16 consecutive keys per 32-key block: row max and row sum
// are lane-local plus one exchange between the two lane halves, and the
// lane's 16 spd bytes are one 16-byte load. P^T then feeds O^T += V^T P^T
// straight from registers. K (row-major) and V^T tiles are staged in LDS and
// shared by the 4 waves; the per-head table (times log2 e) lives in LDS.
#include "common.hpp"
#include "kernels.hpp"

namespace gt {

namespace {

constexpr int kWaves = 4;
constexpr int kBC = 64;          // keys per LDS tile

template <int D, int QB, bool OUT_F32>
__global__ __launch_bounds__(256) void fwd_bf16_kernel(FwdArgs a) {
  constexpr int KB = kBC / 32;   // 32-key sub-blocks per tile
  constexpr int NKC = D / 16;    // k-chunks of Q K^T
  constexpr int NCB = D / 32;    // 32-row blocks of O^T
  constexpr int CPR = D / 8;     // 16-byte chunks per K row
  constexpr int BR = kWaves * 32 * QB;

  __shared__ __attribute__((aligned(16))) uint16_t sK[kBC * D];
  __shared__ __attribute__((aligned(16))) uint16_t sV[D * kBC];   // V^T
  __shared__ float sT[256];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, g = lane >> 5;

  const int64_t nqb = (a.Sq + BR - 1) / BR;
  const int64_t lid = xcd_remap(blockIdx.x, nqb * a.H);
  const int h = (int)(lid % a.H);
  const int64_t qblk = lid / a.H;
  const int64_t qbase = qblk * BR + (int64_t)wave * 32 * QB;

  for (int t = tid; t < 256; t += 256)
    sT[t] = (t < a.n_buckets) ? a.table[(int64_t)h * a.n_buckets + t] * kLog2e : 0.0f;

  const uint16_t* qh = reinterpret_cast<const uint16_t*>(a.q) + (int64_t)h * a.Sq * D;
  const uint16_t* kh = reinterpret_cast<const uint16_t*>(a.k) + (int64_t)h * a.Sk * D;
  const uint16_t* vh = reinterpret_cast<const uint16_t*>(a.v) + (int64_t)h * a.Sk * D;
  const float sl2 = a.scale * kLog2e;

  bf16x8 qf[QB][NKC];
  const uint8_t* srow[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int64_t i = qbase + qb * 32 + col;
    const bool ok = i < a.Sq;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc)
      qf[qb][kc] = ok ? *reinterpret_cast<const bf16x8*>(qh + i * D + kc * 16 + g * 8)
                      : zero_bf16x8();
    srow[qb] = ok ? a.spd + (a.row_off + i) * a.ld_spd + a.col_off : nullptr;
  }

  float m[QB], l[QB];
  f32x16 acc[QB][NCB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    m[qb] = -INFINITY;
    l[qb] = 0.0f;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[qb][cb] = zero_f32x16();
  }

  for (int64_t j0 = 0; j0 < a.Sk; j0 += kBC) {
    __syncthreads();
    // K tile, row-major with swizzled 16-byte chunks.
    for (int c = tid; c < kBC * CPR; c += 256) {
      const int row = c / CPR, ch = c % CPR;
      uint4 val = make_uint4(0, 0, 0, 0);
      if (j0 + row < a.Sk) val = *reinterpret_cast<const uint4*>(kh + (j0 + row) * D + ch * 8);
      *reinterpret_cast<uint4*>(sK + row * D + swz_rows<D>(row, ch) * 8) = val;
    }
    // V^T tile: two key rows per thread packed into dwords.
    for (int c = tid; c < (kBC / 2) * CPR; c += 256) {
      const int jp = c % (kBC / 2), cc = c / (kBC / 2);
      const int j = 2 * jp;
      uint4 v0 = make_uint4(0, 0, 0, 0), v1 = make_uint4(0, 0, 0, 0);
      if (j0 + j < a.Sk) v0 = *reinterpret_cast<const uint4*>(vh + (j0 + j) * D + cc * 8);
      if (j0 + j + 1 < a.Sk) v1 = *reinterpret_cast<const uint4*>(vh + (j0 + j + 1) * D + cc * 8);
      const uint16_t* p0 = reinterpret_cast<const uint16_t*>(&v0);
      const uint16_t* p1 = reinterpret_cast<const uint16_t*>(&v1);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int crow = cc * 8 + e;
        const uint32_t w = (uint32_t)p0[e] | ((uint32_t)p1[e] << 16);
        *reinterpret_cast<uint32_t*>(sV + crow * kBC + swz_t64(crow, j >> 3) * 8 + (j & 7)) = w;
      }
    }
    __syncthreads();

#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float x[KB][16];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        f32x16 s = zero_f32x16();
        const int krow = kb * 32 + perm32(col);
#pragma unroll
        for (int kc = 0; kc < NKC; ++kc)
          s = mfma32(lds_b128(sK + krow * D + swz_rows<D>(krow, kc * 2 + g) * 8), qf[qb][kc], s);
        const int64_t jb = j0 + kb * 32 + 16 * g;
        uint32_t w4[4];
        load_spd16(srow[qb], jb, a.Sk, a.spd_vec != 0, w4);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const uint32_t b = (w4[r >> 2] >> (8 * (r & 3))) & 0xffu;
          const float xv = s[r] * sl2 + sT[b];
          x[kb][r] = (jb + r < a.Sk) ? xv : -INFINITY;
        }
      }
      float mx = x[0][0];
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, x[kb][r]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float mnew = fmaxf(m[qb], mx);
      const float msafe = (mnew == -INFINITY) ? 0.0f : mnew;
      const float alpha = exp2_fast(m[qb] - msafe);
      m[qb] = mnew;
      l[qb] *= alpha;
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[qb][cb][r] *= alpha;
      float ls = 0.0f;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        float p[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          p[r] = exp2_fast(x[kb][r] - msafe);
          ls += p[r];
        }
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const bf16x8 pb = cvt_bf16x8(p + 8 * q);
#pragma unroll
          for (int cb = 0; cb < NCB; ++cb) {
            const int crow = cb * 32 + col;
            const bf16x8 vf = lds_b128(sV + crow * kBC + swz_t64(crow, kb * 4 + 2 * g + q) * 8);
            acc[qb][cb] = mfma32(vf, pb, acc[qb][cb]);
          }
        }
      }
      l[qb] += ls;
    }
  }

  // Epilogue: O = O_acc / l, LSE = (m + log2 l) ln 2.
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float lt = l[qb] + __shfl_xor(l[qb], 32);
    const int64_t i = qbase + qb * 32 + col;
    if (i >= a.Sq) continue;
    const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = cb * 32 + 8 * u + 4 * g;
        const float o0 = acc[qb][cb][4 * u + 0] * inv, o1 = acc[qb][cb][4 * u + 1] * inv;
        const float o2 = acc[qb][cb][4 * u + 2] * inv, o3 = acc[qb][cb][4 * u + 3] * inv;
        if constexpr (OUT_F32) {
          float* op = reinterpret_cast<float*>(a.o) + ((int64_t)h * a.Sq + i) * D + c;
          *reinterpret_cast<float4*>(op) = make_float4(o0, o1, o2, o3);
        } else {
          uint16_t* op = reinterpret_cast<uint16_t*>(a.o) + ((int64_t)h * a.Sq + i) * D + c;
          uint2 pk;
          pk.x = (uint32_t)f2bf(o0) | ((uint32_t)f2bf(o1) << 16);
          pk.y = (uint32_t)f2bf(o2) | ((uint32_t)f2bf(o3) << 16);
          *reinterpret_cast<uint2*>(op) = pk;
        }
      }
    }
    if (g == 0)
      a.lse[(int64_t)h * a.Sq + i] = lt > 0.0f ? (m[qb] + __log2f(lt)) * kLn2 : -INFINITY;
  }
}

// fp32 path: one thread per query row, keys staged through LDS, exact fp32
// math with expf/logf. Written for the small fp32 workloads.
template <int D>
__global__ __launch_bounds__(128) void fwd_f32_kernel(FwdArgs a) {
  constexpr int TK = 32;
  __shared__ float sK[TK][D];
  __shared__ float sV[TK][D];
  __shared__ float sT[256];
  const int tid = threadIdx.x;
  const int64_t nqb = (a.Sq + 127) / 128;
  const int h = (int)(blockIdx.x / nqb);
  const int64_t i = (blockIdx.x % nqb) * 128 + tid;
  for (int t = tid; t < 256; t += 128)
    sT[t] = (t < a.n_buckets) ? a.table[(int64_t)h * a.n_buckets + t] : 0.0f;
  const float* qh = reinterpret_cast<const float*>(a.q) + (int64_t)h * a.Sq * D;
  const float* kh = reinterpret_cast<const float*>(a.k) + (int64_t)h * a.Sk * D;
  const float* vh = reinterpret_cast<const float*>(a.v) + (int64_t)h * a.Sk * D;
  const bool ok = i < a.Sq;
  float qv[D], acc[D];
#pragma unroll
  for (int c = 0; c < D; ++c) {
    qv[c] = ok ? qh[i * D + c] * a.scale : 0.0f;
    acc[c] = 0.0f;
  }
  const uint8_t* srow = ok ? a.spd + (a.row_off + i) * a.ld_spd + a.col_off : nullptr;
  float m = -INFINITY, l = 0.0f;
  for (int64_t j0 = 0; j0 < a.Sk; j0 += TK) {
    __syncthreads();
    for (int t = tid; t < TK * D; t += 128) {
      const int r = t / D, c = t % D;
      const bool in = j0 + r < a.Sk;
      sK[r][c] = in ? kh[(j0 + r) * D + c] : 0.0f;
      sV[r][c] = in ? vh[(j0 + r) * D + c] : 0.0f;
    }
    __syncthreads();
    if (!ok) continue;
    const int nk = (int)((a.Sk - j0) < TK ? (a.Sk - j0) : TK);
    for (int r = 0; r < nk; ++r) {
      float s = 0.0f;
#pragma unroll
      for (int c = 0; c < D; ++c) s = fmaf(qv[c], sK[r][c], s);
      s += sT[srow[j0 + r]];
      if (s == -INFINITY) continue;
      if (s > m) {
        const float alpha = (m == -INFINITY) ? 0.0f : expf(m - s);
        l *= alpha;
#pragma unroll
        for (int c = 0; c < D; ++c) acc[c] *= alpha;
        m = s;
      }
      const float p = expf(s - m);
      l += p;
#pragma unroll
      for (int c = 0; c < D; ++c) acc[c] = fmaf(p, sV[r][c], acc[c]);
    }
  }
  if (!ok) return;
  const float inv = l > 0.0f ? 1.0f / l : 0.0f;
  float* op = reinterpret_cast<float*>(a.o) + ((int64_t)h * a.Sq + i) * D;
#pragma unroll
  for (int c = 0; c < D; ++c) op[c] = acc[c] * inv;
  a.lse[(int64_t)h * a.Sq + i] = l > 0.0f ? m + logf(l) : -INFINITY;
}

template <int D, int QB, bool OUT_F32>
hipError_t launch_fwd_bf16(const FwdArgs& a, hipStream_t s) {
  constexpr int BR = kWaves * 32 * QB;
  const int64_t nqb = (a.Sq + BR - 1) / BR;
  const int64_t grid = nqb * a.H;
  hipLaunchKernelGGL((fwd_bf16_kernel<D, QB, OUT_F32>), dim3((unsigned)grid), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_fwd_f32(const FwdArgs& a, hipStream_t s) {
  const int64_t nqb = (a.Sq + 127) / 128;
  hipLaunchKernelGGL((fwd_f32_kernel<D>), dim3((unsigned)(nqb * a.H)), dim3(128), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_fwd(const FwdArgs& a, int d, bool bf16, bool out_f32, hipStream_t s) {
  if (bf16) {
    if (d == 64) return out_f32 ? launch_fwd_bf16<64, 1, true>(a, s) : launch_fwd_bf16<64, 1, false>(a, s);
    return out_f32 ? launch_fwd_bf16<32, 1, true>(a, s) : launch_fwd_bf16<32, 1, false>(a, s);
  }
  return d == 64 ? launch_fwd_f32<64>(a, s) : launch_fwd_f32<32>(a, s);
}

}  // namespace gt
