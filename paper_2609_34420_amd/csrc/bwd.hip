// Backward kernels of biased attention.
//
// With P = softmax(S), S = scale Q K^T + B (Eq. (1)) and L = sum(O * dO):
//   Dlt_i = sum_c dO_ic O_ic,  dS = P * (dO V^T - Dlt),
//   dV = P^T dO,  dK = scale dS^T Q,  dQ = scale dS K,
//   dtable[h, b] = sum of dS_ij over pairs with spd_ij = b.
// P is recomputed from the saved LSE, never stored.
//
// bf16 path, three launches:
//   prep  : lse2 = LSE log2(e) (+inf for an empty row, so P = 0), Dlt; zero dtable
//   dkdv  : key-stationary; each wave owns 32 keys, S = Q K^T with lanes on
//           keys, so P and dS feed dV^T += dO^T P and dK^T += Q^T dS from
//           registers; the dS of every pair is also scattered into an LDS
//           histogram by spd bucket, flushed once per workgroup with one
//           global atomic per bucket
//   dq    : query-stationary; S^T = K Q^T with lanes on queries (as in the
//           forward), dQ^T += K^T dS^T.
// Splitting dQ from dK/dV recomputes two products but needs no atomics on
// dQ.
#include "common.hpp"
#include "kernels.hpp"

namespace gt {

namespace {

constexpr int kWaves = 4;

// ---------------------------------------------------------------------------
// Preprocess: lse2, Dlt; dtable = 0.
// ---------------------------------------------------------------------------
template <int D, bool BF16>
__global__ __launch_bounds__(256) void bwd_prep_kernel(BwdArgs a) {
  const int64_t row = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (blockIdx.x == 0) {
    for (int t = threadIdx.x; t < a.H * a.n_buckets; t += 256) a.dtable[t] = 0.0f;
  }
  if (row >= (int64_t)a.H * a.N) return;
  float acc = 0.0f;
  if constexpr (BF16) {
    const uint16_t* o = reinterpret_cast<const uint16_t*>(a.o) + row * D;
    const uint16_t* d = reinterpret_cast<const uint16_t*>(a.d_o) + row * D;
#pragma unroll
    for (int c = 0; c < D; c += 8) {
      const uint4 ov = *reinterpret_cast<const uint4*>(o + c);
      const uint4 dv = *reinterpret_cast<const uint4*>(d + c);
      const uint16_t* op = reinterpret_cast<const uint16_t*>(&ov);
      const uint16_t* dp = reinterpret_cast<const uint16_t*>(&dv);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc = fmaf(bf2f(op[e]), bf2f(dp[e]), acc);
    }
  } else {
    const float* o = reinterpret_cast<const float*>(a.o) + row * D;
    const float* d = reinterpret_cast<const float*>(a.d_o) + row * D;
#pragma unroll
    for (int c = 0; c < D; ++c) acc = fmaf(o[c], d[c], acc);
  }
  a.dlt[row] = acc;
  const float L = a.lse[row];
  a.lse2[row] = (L == -INFINITY) ? INFINITY : L * kLog2e;
}

// ---------------------------------------------------------------------------
// bf16 dK / dV / dtable: key-stationary.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void bwd_dkdv_bf16_kernel(BwdArgs a) {
  constexpr int BQ = 64;         // queries per LDS tile
  constexpr int NKC = D / 16;
  constexpr int NCB = D / 32;
  constexpr int CPR = D / 8;
  constexpr int BK = kWaves * 32;  // keys per workgroup

  __shared__ __attribute__((aligned(16))) uint16_t sQ[BQ * D];
  __shared__ __attribute__((aligned(16))) uint16_t sO[BQ * D];    // dO
  __shared__ __attribute__((aligned(16))) uint16_t sQt[D * BQ];   // Q^T
  __shared__ __attribute__((aligned(16))) uint16_t sOt[D * BQ];   // dO^T
  __shared__ __attribute__((aligned(16))) float sL[BQ];
  __shared__ __attribute__((aligned(16))) float sD[BQ];
  __shared__ float sT[256];
  __shared__ float sH[256 * 32];   // bucket histogram, 32 copies

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, g = lane >> 5;

  const int64_t nkb = (a.N + BK - 1) / BK;
  const int64_t lid = xcd_remap(blockIdx.x, nkb * a.H);
  const int h = (int)(lid % a.H);
  const int64_t kblk = lid / a.H;
  const int64_t j = kblk * BK + wave * 32 + col;   // this lane's key
  const bool jok = j < a.N;

  for (int t = tid; t < 256; t += 256)
    sT[t] = (t < a.n_buckets) ? a.table[(int64_t)h * a.n_buckets + t] * kLog2e : 0.0f;
  for (int t = tid; t < 256 * 32; t += 256) sH[t] = 0.0f;

  const int64_t hoff = (int64_t)h * a.N * D;
  const uint16_t* qh = reinterpret_cast<const uint16_t*>(a.q) + hoff;
  const uint16_t* kh = reinterpret_cast<const uint16_t*>(a.k) + hoff;
  const uint16_t* vh = reinterpret_cast<const uint16_t*>(a.v) + hoff;
  const uint16_t* oh = reinterpret_cast<const uint16_t*>(a.d_o) + hoff;
  const float* lse2h = a.lse2 + (int64_t)h * a.N;
  const float* dlth = a.dlt + (int64_t)h * a.N;
  const float sl2 = a.scale * kLog2e;

  bf16x8 kf[NKC], vf[NKC];
#pragma unroll
  for (int kc = 0; kc < NKC; ++kc) {
    kf[kc] = jok ? *reinterpret_cast<const bf16x8*>(kh + j * D + kc * 16 + g * 8) : zero_bf16x8();
    vf[kc] = jok ? *reinterpret_cast<const bf16x8*>(vh + j * D + kc * 16 + g * 8) : zero_bf16x8();
  }
  f32x16 dk[NCB], dv[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    dk[cb] = zero_f32x16();
    dv[cb] = zero_f32x16();
  }
  const uint8_t* scol = a.spd + (jok ? j : 0);

  for (int64_t i0 = 0; i0 < a.N; i0 += BQ) {
    __syncthreads();
    // Q, dO row-major (swizzled); Q^T, dO^T transposed (swizzled).
    for (int c = tid; c < BQ * CPR; c += 256) {
      const int row = c / CPR, ch = c % CPR;
      uint4 qv = make_uint4(0, 0, 0, 0), dv4 = make_uint4(0, 0, 0, 0);
      if (i0 + row < a.N) {
        qv = *reinterpret_cast<const uint4*>(qh + (i0 + row) * D + ch * 8);
        dv4 = *reinterpret_cast<const uint4*>(oh + (i0 + row) * D + ch * 8);
      }
      *reinterpret_cast<uint4*>(sQ + row * D + swz_rows<D>(row, ch) * 8) = qv;
      *reinterpret_cast<uint4*>(sO + row * D + swz_rows<D>(row, ch) * 8) = dv4;
    }
    for (int c = tid; c < (BQ / 2) * CPR; c += 256) {
      const int ip = c % (BQ / 2), cc = c / (BQ / 2);
      const int i = 2 * ip;
      uint4 q0 = make_uint4(0, 0, 0, 0), q1 = q0, d0 = q0, d1 = q0;
      if (i0 + i < a.N) {
        q0 = *reinterpret_cast<const uint4*>(qh + (i0 + i) * D + cc * 8);
        d0 = *reinterpret_cast<const uint4*>(oh + (i0 + i) * D + cc * 8);
      }
      if (i0 + i + 1 < a.N) {
        q1 = *reinterpret_cast<const uint4*>(qh + (i0 + i + 1) * D + cc * 8);
        d1 = *reinterpret_cast<const uint4*>(oh + (i0 + i + 1) * D + cc * 8);
      }
      const uint16_t* pq0 = reinterpret_cast<const uint16_t*>(&q0);
      const uint16_t* pq1 = reinterpret_cast<const uint16_t*>(&q1);
      const uint16_t* pd0 = reinterpret_cast<const uint16_t*>(&d0);
      const uint16_t* pd1 = reinterpret_cast<const uint16_t*>(&d1);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int crow = cc * 8 + e;
        const int off = crow * BQ + swz_t64(crow, i >> 3) * 8 + (i & 7);
        *reinterpret_cast<uint32_t*>(sQt + off) = (uint32_t)pq0[e] | ((uint32_t)pq1[e] << 16);
        *reinterpret_cast<uint32_t*>(sOt + off) = (uint32_t)pd0[e] | ((uint32_t)pd1[e] << 16);
      }
    }
    for (int t = tid; t < BQ; t += 256) {
      const bool in = i0 + t < a.N;
      sL[t] = in ? lse2h[i0 + t] : INFINITY;   // padded rows: P = 0
      sD[t] = in ? dlth[i0 + t] : 0.0f;
    }
    __syncthreads();

#pragma unroll
    for (int qs = 0; qs < BQ / 32; ++qs) {
      f32x16 s = zero_f32x16(), dp = zero_f32x16();
      const int qrow = qs * 32 + perm32(col);
#pragma unroll
      for (int kc = 0; kc < NKC; ++kc) {
        const int off = qrow * D + swz_rows<D>(qrow, kc * 2 + g) * 8;
        s = mfma32(lds_b128(sQ + off), kf[kc], s);
        dp = mfma32(lds_b128(sO + off), vf[kc], dp);
      }
      // Lane: key j; registers r: queries i0 + qs*32 + 16 g + r.
      const int ib = qs * 32 + 16 * g;
      float p[16], ds[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t i = i0 + ib + r;
        const uint32_t b = (jok && i < a.N) ? (uint32_t)scol[i * a.ld_spd] : 0u;
        const float x = s[r] * sl2 + sT[b] - sL[ib + r];
        const float pv = jok ? exp2_fast(x) : 0.0f;
        p[r] = pv;
        ds[r] = pv * (dp[r] - sD[ib + r]);
        atomicAdd(&sH[b * 32 + col], ds[r]);
      }
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const bf16x8 pb = cvt_bf16x8(p + 8 * q);
        const bf16x8 db = cvt_bf16x8(ds + 8 * q);
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
          const int crow = cb * 32 + col;
          const int off = crow * BQ + swz_t64(crow, (ib >> 3) + q) * 8;
          dv[cb] = mfma32(lds_b128(sOt + off), pb, dv[cb]);
          dk[cb] = mfma32(lds_b128(sQt + off), db, dk[cb]);
        }
      }
    }
  }

  // dK = scale dK^T^T, dV: lane (key j) holds features cb*32 + 8u + 4g + t.
  if (jok) {
    uint16_t* dkp = reinterpret_cast<uint16_t*>(a.dk) + hoff + j * D;
    uint16_t* dvp = reinterpret_cast<uint16_t*>(a.dv) + hoff + j * D;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = cb * 32 + 8 * u + 4 * g;
        uint2 pk, pv;
        pk.x = (uint32_t)f2bf(dk[cb][4 * u] * a.scale) | ((uint32_t)f2bf(dk[cb][4 * u + 1] * a.scale) << 16);
        pk.y = (uint32_t)f2bf(dk[cb][4 * u + 2] * a.scale) | ((uint32_t)f2bf(dk[cb][4 * u + 3] * a.scale) << 16);
        pv.x = (uint32_t)f2bf(dv[cb][4 * u]) | ((uint32_t)f2bf(dv[cb][4 * u + 1]) << 16);
        pv.y = (uint32_t)f2bf(dv[cb][4 * u + 2]) | ((uint32_t)f2bf(dv[cb][4 * u + 3]) << 16);
        *reinterpret_cast<uint2*>(dkp + c) = pk;
        *reinterpret_cast<uint2*>(dvp + c) = pv;
      }
    }
  }
  __syncthreads();
  for (int b = tid; b < a.n_buckets; b += 256) {
    float t = 0.0f;
    for (int c = 0; c < 32; ++c) t += sH[b * 32 + ((c + b) & 31)];
    if (t != 0.0f) atomicAdd(&a.dtable[(int64_t)h * a.n_buckets + b], t);
  }
}

// ---------------------------------------------------------------------------
// bf16 dQ: query-stationary, S^T = K Q^T (lanes on queries).
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(256) void bwd_dq_bf16_kernel(BwdArgs a) {
  constexpr int BC = 64;
  constexpr int KB = BC / 32;
  constexpr int NKC = D / 16;
  constexpr int NCB = D / 32;
  constexpr int CPR = D / 8;
  constexpr int BR = kWaves * 32;

  __shared__ __attribute__((aligned(16))) uint16_t sK[BC * D];
  __shared__ __attribute__((aligned(16))) uint16_t sV[BC * D];
  __shared__ __attribute__((aligned(16))) uint16_t sKt[D * BC];
  __shared__ float sT[256];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int col = lane & 31, g = lane >> 5;

  const int64_t nqb = (a.N + BR - 1) / BR;
  const int64_t lid = xcd_remap(blockIdx.x, nqb * a.H);
  const int h = (int)(lid % a.H);
  const int64_t qblk = lid / a.H;
  const int64_t i = qblk * BR + wave * 32 + col;   // this lane's query
  const bool iok = i < a.N;

  for (int t = tid; t < 256; t += 256)
    sT[t] = (t < a.n_buckets) ? a.table[(int64_t)h * a.n_buckets + t] * kLog2e : 0.0f;

  const int64_t hoff = (int64_t)h * a.N * D;
  const uint16_t* qh = reinterpret_cast<const uint16_t*>(a.q) + hoff;
  const uint16_t* kh = reinterpret_cast<const uint16_t*>(a.k) + hoff;
  const uint16_t* vh = reinterpret_cast<const uint16_t*>(a.v) + hoff;
  const uint16_t* oh = reinterpret_cast<const uint16_t*>(a.d_o) + hoff;
  const float sl2 = a.scale * kLog2e;

  bf16x8 qf[NKC], df[NKC];
#pragma unroll
  for (int kc = 0; kc < NKC; ++kc) {
    qf[kc] = iok ? *reinterpret_cast<const bf16x8*>(qh + i * D + kc * 16 + g * 8) : zero_bf16x8();
    df[kc] = iok ? *reinterpret_cast<const bf16x8*>(oh + i * D + kc * 16 + g * 8) : zero_bf16x8();
  }
  const float lse2 = iok ? a.lse2[(int64_t)h * a.N + i] : INFINITY;
  const float dlt = iok ? a.dlt[(int64_t)h * a.N + i] : 0.0f;
  const uint8_t* srow = iok ? a.spd + i * a.ld_spd : nullptr;
  f32x16 acc[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) acc[cb] = zero_f32x16();

  for (int64_t j0 = 0; j0 < a.N; j0 += BC) {
    __syncthreads();
    for (int c = tid; c < BC * CPR; c += 256) {
      const int row = c / CPR, ch = c % CPR;
      uint4 kv = make_uint4(0, 0, 0, 0), vv = kv;
      if (j0 + row < a.N) {
        kv = *reinterpret_cast<const uint4*>(kh + (j0 + row) * D + ch * 8);
        vv = *reinterpret_cast<const uint4*>(vh + (j0 + row) * D + ch * 8);
      }
      *reinterpret_cast<uint4*>(sK + row * D + swz_rows<D>(row, ch) * 8) = kv;
      *reinterpret_cast<uint4*>(sV + row * D + swz_rows<D>(row, ch) * 8) = vv;
    }
    for (int c = tid; c < (BC / 2) * CPR; c += 256) {
      const int jp = c % (BC / 2), cc = c / (BC / 2);
      const int jj = 2 * jp;
      uint4 k0 = make_uint4(0, 0, 0, 0), k1 = k0;
      if (j0 + jj < a.N) k0 = *reinterpret_cast<const uint4*>(kh + (j0 + jj) * D + cc * 8);
      if (j0 + jj + 1 < a.N) k1 = *reinterpret_cast<const uint4*>(kh + (j0 + jj + 1) * D + cc * 8);
      const uint16_t* p0 = reinterpret_cast<const uint16_t*>(&k0);
      const uint16_t* p1 = reinterpret_cast<const uint16_t*>(&k1);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int crow = cc * 8 + e;
        *reinterpret_cast<uint32_t*>(sKt + crow * BC + swz_t64(crow, jj >> 3) * 8 + (jj & 7)) =
            (uint32_t)p0[e] | ((uint32_t)p1[e] << 16);
      }
    }
    __syncthreads();

#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      f32x16 s = zero_f32x16(), dp = zero_f32x16();
      const int krow = kb * 32 + perm32(col);
#pragma unroll
      for (int kc = 0; kc < NKC; ++kc) {
        const int off = krow * D + swz_rows<D>(krow, kc * 2 + g) * 8;
        s = mfma32(lds_b128(sK + off), qf[kc], s);
        dp = mfma32(lds_b128(sV + off), df[kc], dp);
      }
      const int64_t jb = j0 + kb * 32 + 16 * g;
      uint32_t w4[4];
      load_spd16(srow, jb, a.N, a.spd_vec != 0, w4);
      float ds[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const uint32_t b = (w4[r >> 2] >> (8 * (r & 3))) & 0xffu;
        const float x = s[r] * sl2 + sT[b] - lse2;
        const float pv = (jb + r < a.N) ? exp2_fast(x) : 0.0f;
        ds[r] = pv * (dp[r] - dlt);
      }
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const bf16x8 db = cvt_bf16x8(ds + 8 * q);
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
          const int crow = cb * 32 + col;
          acc[cb] = mfma32(lds_b128(sKt + crow * BC + swz_t64(crow, kb * 4 + 2 * g + q) * 8), db, acc[cb]);
        }
      }
    }
  }

  if (iok) {
    uint16_t* dqp = reinterpret_cast<uint16_t*>(a.dq) + hoff + i * D;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = cb * 32 + 8 * u + 4 * g;
        uint2 pk;
        pk.x = (uint32_t)f2bf(acc[cb][4 * u] * a.scale) | ((uint32_t)f2bf(acc[cb][4 * u + 1] * a.scale) << 16);
        pk.y = (uint32_t)f2bf(acc[cb][4 * u + 2] * a.scale) | ((uint32_t)f2bf(acc[cb][4 * u + 3] * a.scale) << 16);
        *reinterpret_cast<uint2*>(dqp + c) = pk;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// fp32 path (small workloads): one thread per query row / key column.
// ---------------------------------------------------------------------------
template <int D>
__global__ __launch_bounds__(128) void bwd_dq_f32_kernel(BwdArgs a) {
  constexpr int TK = 32;
  __shared__ float sK[TK][D];
  __shared__ float sV[TK][D];
  __shared__ float sT[256];
  __shared__ float sH[256];
  const int tid = threadIdx.x;
  const int64_t nqb = (a.N + 127) / 128;
  const int h = (int)(blockIdx.x / nqb);
  const int64_t i = (blockIdx.x % nqb) * 128 + tid;
  for (int t = tid; t < 256; t += 128) {
    sT[t] = (t < a.n_buckets) ? a.table[(int64_t)h * a.n_buckets + t] : 0.0f;
    sH[t] = 0.0f;
  }
  const int64_t hoff = (int64_t)h * a.N * D;
  const float* qh = reinterpret_cast<const float*>(a.q) + hoff;
  const float* kh = reinterpret_cast<const float*>(a.k) + hoff;
  const float* vh = reinterpret_cast<const float*>(a.v) + hoff;
  const float* oh = reinterpret_cast<const float*>(a.d_o) + hoff;
  const bool ok = i < a.N;
  float qv[D], dov[D], acc[D];
#pragma unroll
  for (int c = 0; c < D; ++c) {
    qv[c] = ok ? qh[i * D + c] * a.scale : 0.0f;
    dov[c] = ok ? oh[i * D + c] : 0.0f;
    acc[c] = 0.0f;
  }
  const float L = ok ? a.lse[(int64_t)h * a.N + i] : -INFINITY;
  const float dlt = ok ? a.dlt[(int64_t)h * a.N + i] : 0.0f;
  const uint8_t* srow = ok ? a.spd + i * a.ld_spd : nullptr;
  for (int64_t j0 = 0; j0 < a.N; j0 += TK) {
    __syncthreads();
    for (int t = tid; t < TK * D; t += 128) {
      const int r = t / D, c = t % D;
      const bool in = j0 + r < a.N;
      sK[r][c] = in ? kh[(j0 + r) * D + c] : 0.0f;
      sV[r][c] = in ? vh[(j0 + r) * D + c] : 0.0f;
    }
    __syncthreads();
    if (!ok || L == -INFINITY) continue;
    const int nk = (int)((a.N - j0) < TK ? (a.N - j0) : TK);
    for (int r = 0; r < nk; ++r) {
      float s = 0.0f, dp = 0.0f;
#pragma unroll
      for (int c = 0; c < D; ++c) {
        s = fmaf(qv[c], sK[r][c], s);
        dp = fmaf(dov[c], sV[r][c], dp);
      }
      const uint32_t b = srow[j0 + r];
      const float p = expf(s + sT[b] - L);
      const float ds = p * (dp - dlt);
#pragma unroll
      for (int c = 0; c < D; ++c) acc[c] = fmaf(ds, sK[r][c], acc[c]);
      if (b < (uint32_t)a.n_buckets) atomicAdd(&sH[b], ds);
    }
  }
  if (ok) {
    float* dqp = reinterpret_cast<float*>(a.dq) + hoff + i * D;
#pragma unroll
    for (int c = 0; c < D; ++c) dqp[c] = acc[c] * a.scale;
  }
  __syncthreads();
  for (int t = tid; t < a.n_buckets; t += 128)
    if (sH[t] != 0.0f) atomicAdd(&a.dtable[(int64_t)h * a.n_buckets + t], sH[t]);
}

template <int D>
__global__ __launch_bounds__(128) void bwd_dkdv_f32_kernel(BwdArgs a) {
  constexpr int TQ = 32;
  __shared__ float sQ[TQ][D];
  __shared__ float sO[TQ][D];
  __shared__ float sL[TQ], sD[TQ];
  __shared__ float sT[256];
  const int tid = threadIdx.x;
  const int64_t nkb = (a.N + 127) / 128;
  const int h = (int)(blockIdx.x / nkb);
  const int64_t j = (blockIdx.x % nkb) * 128 + tid;
  for (int t = tid; t < 256; t += 128)
    sT[t] = (t < a.n_buckets) ? a.table[(int64_t)h * a.n_buckets + t] : 0.0f;
  const int64_t hoff = (int64_t)h * a.N * D;
  const float* qh = reinterpret_cast<const float*>(a.q) + hoff;
  const float* kh = reinterpret_cast<const float*>(a.k) + hoff;
  const float* vh = reinterpret_cast<const float*>(a.v) + hoff;
  const float* oh = reinterpret_cast<const float*>(a.d_o) + hoff;
  const bool ok = j < a.N;
  float kv[D], vv[D], dk[D], dv[D];
#pragma unroll
  for (int c = 0; c < D; ++c) {
    kv[c] = ok ? kh[j * D + c] * a.scale : 0.0f;
    vv[c] = ok ? vh[j * D + c] : 0.0f;
    dk[c] = 0.0f;
    dv[c] = 0.0f;
  }
  for (int64_t i0 = 0; i0 < a.N; i0 += TQ) {
    __syncthreads();
    for (int t = tid; t < TQ * D; t += 128) {
      const int r = t / D, c = t % D;
      const bool in = i0 + r < a.N;
      sQ[r][c] = in ? qh[(i0 + r) * D + c] : 0.0f;
      sO[r][c] = in ? oh[(i0 + r) * D + c] : 0.0f;
    }
    for (int t = tid; t < TQ; t += 128) {
      const bool in = i0 + t < a.N;
      sL[t] = in ? a.lse[(int64_t)h * a.N + i0 + t] : -INFINITY;
      sD[t] = in ? a.dlt[(int64_t)h * a.N + i0 + t] : 0.0f;
    }
    __syncthreads();
    if (!ok) continue;
    const int nq = (int)((a.N - i0) < TQ ? (a.N - i0) : TQ);
    for (int r = 0; r < nq; ++r) {
      if (sL[r] == -INFINITY) continue;
      float s = 0.0f, dp = 0.0f;
#pragma unroll
      for (int c = 0; c < D; ++c) {
        s = fmaf(sQ[r][c], kv[c], s);
        dp = fmaf(sO[r][c], vv[c], dp);
      }
      const float p = expf(s + sT[a.spd[(i0 + r) * a.ld_spd + j]] - sL[r]);
      const float ds = p * (dp - sD[r]);
#pragma unroll
      for (int c = 0; c < D; ++c) {
        dv[c] = fmaf(p, sO[r][c], dv[c]);
        dk[c] = fmaf(ds, sQ[r][c], dk[c]);
      }
    }
  }
  if (!ok) return;
  float* dkp = reinterpret_cast<float*>(a.dk) + hoff + j * D;
  float* dvp = reinterpret_cast<float*>(a.dv) + hoff + j * D;
#pragma unroll
  for (int c = 0; c < D; ++c) {
    dkp[c] = dk[c] * a.scale;
    dvp[c] = dv[c];
  }
}

template <int D>
hipError_t launch_bwd_t(const BwdArgs& a, bool bf16, hipStream_t s) {
  const int64_t rows = (int64_t)a.H * a.N;
  if (bf16)
    hipLaunchKernelGGL((bwd_prep_kernel<D, true>), dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL((bwd_prep_kernel<D, false>), dim3((unsigned)((rows + 255) / 256)), dim3(256), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (bf16) {
    const int64_t nkb = (a.N + kWaves * 32 - 1) / (kWaves * 32);
    hipLaunchKernelGGL((bwd_dkdv_bf16_kernel<D>), dim3((unsigned)(nkb * a.H)), dim3(256), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const int64_t nqb = (a.N + kWaves * 32 - 1) / (kWaves * 32);
    hipLaunchKernelGGL((bwd_dq_bf16_kernel<D>), dim3((unsigned)(nqb * a.H)), dim3(256), 0, s, a);
    return hipGetLastError();
  }
  const int64_t nb = (a.N + 127) / 128;
  hipLaunchKernelGGL((bwd_dkdv_f32_kernel<D>), dim3((unsigned)(nb * a.H)), dim3(128), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL((bwd_dq_f32_kernel<D>), dim3((unsigned)(nb * a.H)), dim3(128), 0, s, a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_bwd(const BwdArgs& a, int d, bool bf16, hipStream_t s) {
  return d == 64 ? launch_bwd_t<64>(a, bf16, s) : launch_bwd_t<32>(a, bf16, s);
}

}  // namespace gt
