// Backward, query-stationary stage: dQ (bf16).
//
// Same layout as the forward: each wave owns 32*QB queries, computes
// S^T = K Q^T and dP^T = V dO^T with the queries on the lanes, forms
// dS^T = P^T * (dP^T - Dlt) from the saved log-sum-exp, and accumulates
// dQ^T += K^T dS^T with dS^T straight from registers. K and V tiles are
// double buffered row-major in LDS (K^T is read with transposing LDS reads)
// and the next tile's global loads and spd bytes are in flight while the
// current one computes.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "stage.hpp"

namespace gt {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kBC = 64;

// One key tile for every query block of the wave. The accumulators of S^T
// and dP^T start at -lse2 / (scale log2 e) and -Dlt, so per score element the
// vector work is the bias FMA, exp2, one multiply and the bf16 conversion.
// Per-lane LDS element offsets (tile-relative; 32-key block and 8-key step
// offsets are immediates). K and V rows share one pattern.
template <int D>
struct DqOffsets {
  int row[D / 16];        // rows perm32(lane), feature chunk 2 kc + g
  int kt[2][D / 32];      // transposing reads h = 0, 1 of K, feature block cb
  __device__ __forceinline__ DqOffsets() {
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) row[kc] = row_operand_off<D>(kc);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int cb = 0; cb < D / 32; ++cb) kt[h][cb] = tr_operand_off<D>(h, cb);
  }
};

// One key tile for every query block of the wave. The accumulators of S^T
// and dP^T start at -lse2 / (scale log2 e) and -Dlt, so per score element the
// vector work is the bias FMA, exp2, one multiply and the bf16 conversion.
template <int D, int QB, bool MASK>
__device__ __forceinline__ void dq_tile(const uint16_t* sK, const uint16_t* sV, const float* sT,
                                        const DqOffsets<D>& off, const bf16x8 (&qf)[QB][D / 16],
                                        const bf16x8 (&df)[QB][D / 16], const f32x16 (&init_s)[QB],
                                        const f32x16 (&init_p)[QB],
                                        const uint32_t (&w)[QB][kBC / 32][4], int64_t j0,
                                        int64_t nk, float sl2, f32x16 (&acc)[QB][D / 32]) {
  constexpr int KB = kBC / 32;
  constexpr int NKC = D / 16;
  constexpr int NCB = D / 32;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 5;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      float tb[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) tb[r] = sT[(w[qb][kb][r >> 2] >> (8 * (r & 3))) & 0xffu];
      f32x16 s = init_s[qb], dp = init_p[qb];
#pragma unroll
      for (int kc = 0; kc < NKC; ++kc) {
        s = mfma32(lds_b128(sK + kb * 32 * D + off.row[kc]), qf[qb][kc], s);
        dp = mfma32(lds_b128(sV + kb * 32 * D + off.row[kc]), df[qb][kc], dp);
      }
      float ds[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float pv = exp2_fast(fmaf(s[r], sl2, tb[r]));
        if constexpr (MASK) pv = (j0 + kb * 32 + 16 * g + r < nk) ? pv : 0.0f;
        ds[r] = pv * dp[r];
      }
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        const bf16x8 db = cvt_bf16x8(ds + 8 * q);
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
          const uint16_t* kt = sK + (kb * 32 + 8 * q) * D;
          acc[qb][cb] = mfma32(lds_tr_operand(kt, off.kt[0][cb], off.kt[1][cb]), db, acc[qb][cb]);
        }
      }
    }
  }
}

// VEC: spd rows are 16-byte aligned. FULL: VEC and N a multiple of the key
// tile, so every spd group is loaded whole and no tile needs masking.
template <int D, int QB, bool VEC, bool FULL>
__global__ __launch_bounds__(kThreads, 2) void bwd_dq_bf16_kernel(BwdArgs a) {
  constexpr int KB = kBC / 32;
  constexpr int NKC = D / 16;
  constexpr int NCB = D / 32;
  constexpr int BR = kWaves * 32 * QB;
  using Stage = RowStage<D, kThreads>;
  static_assert(kBC == kTileRows, "key tile is one staged tile");

  __shared__ __attribute__((aligned(16))) uint16_t sK[2][kBC * D];
  __shared__ __attribute__((aligned(16))) uint16_t sV[2][kBC * D];
  __shared__ float sT[256];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = wave_id();
  const int col = lane & 31, g = lane >> 5;

  const int64_t nqb = (a.Sq + BR - 1) / BR;
  const int64_t lid = xcd_remap(blockIdx.x, nqb * a.H);
  const int h = (int)(lid % a.H);
  const int64_t qblk = lid / a.H;
  const int64_t qbase = qblk * BR + (int64_t)wave * 32 * QB;

  for (int t = tid; t < 256; t += kThreads)
    sT[t] = (t < a.n_buckets) ? a.table[(int64_t)h * a.n_buckets + t] * kLog2e : 0.0f;

  const int64_t hq = (int64_t)h * a.Sq * D;   // query-side rows
  const int64_t hk = (int64_t)h * a.Sk * D;   // key-side rows
  const uint16_t* qh = reinterpret_cast<const uint16_t*>(a.q) + hq;
  const uint16_t* kh = reinterpret_cast<const uint16_t*>(a.k) + hk;
  const uint16_t* vh = reinterpret_cast<const uint16_t*>(a.v) + hk;
  const uint16_t* oh = reinterpret_cast<const uint16_t*>(a.d_o) + hq;
  const float sl2 = a.scale * kLog2e;

  // Q^T, dO^T operands and statistics; rows past N load the clamped row N-1
  // and get lse2 = +inf (P = 0); their dQ is not stored.
  bf16x8 qf[QB][NKC], df[QB][NKC];
  f32x16 init_s[QB], init_p[QB];
  int64_t qrow[QB];
  const float inv_sl2 = 1.0f / sl2;
  f32x16 acc[QB][NCB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int64_t i = qbase + qb * 32 + col;
    qrow[qb] = i < a.Sq ? i : a.Sq - 1;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      qf[qb][kc] = *reinterpret_cast<const bf16x8*>(qh + qrow[qb] * D + kc * 16 + g * 8);
      df[qb][kc] = *reinterpret_cast<const bf16x8*>(oh + qrow[qb] * D + kc * 16 + g * 8);
    }
    const float l2 = a.lse2[(int64_t)h * a.Sq + qrow[qb]];
    const float dl = a.dlt[(int64_t)h * a.Sq + qrow[qb]];
    const float is = i < a.Sq ? -l2 * inv_sl2 : -INFINITY;   // padded rows: P = 0
    const float ip = i < a.Sq ? -dl : 0.0f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      init_s[qb][r] = is;
      init_p[qb][r] = ip;
    }
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[qb][cb] = zero_f32x16();
  }

  const int64_t ld = a.ld_spd;
  const int64_t rb = qbase < a.Sq ? qbase : a.Sq - 1;
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(a.spd + (a.row_off + rb) * ld + a.col_off);
  uint32_t voff[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) voff[qb] = (uint32_t)((qrow[qb] - rb) * ld) + 16u * g;
  auto fetch_spd = [&](int64_t jt, uint32_t (&w)[QB][KB][4]) {
    if (FULL || (VEC && jt + kBC <= a.Sk)) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) buf_u128(rs, voff[qb], (uint32_t)(jt + kb * 32), w[qb][kb]);
    } else {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const uint8_t* row = a.spd + (a.row_off + qrow[qb]) * ld + a.col_off;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) load_spd16_bytes(row, jt + kb * 32 + 16 * g, a.Sk, w[qb][kb]);
      }
    }
  };

  const int64_t ntiles = (a.Sk + kBC - 1) / kBC;
  const DqOffsets<D> off;
  Stage stK, stV;
  uint32_t wA[QB][KB][4], wB[QB][KB][4];   // spd words of even / odd tiles
  stK.load(tile_rsrc<D>(kh, 0, a.Sk));
  stV.load(tile_rsrc<D>(vh, 0, a.Sk));
  fetch_spd(0, wA);
  stK.store(sK[0]);
  stV.store(sV[0]);
  wait_loads();
  __syncthreads();

  // One key tile: prefetch the next (the last tile re-reads itself, so the
  // loads in flight are the same on every path), compute on buffer BUF,
  // stage the prefetch into the other buffer.
  auto step = [&](int64_t t, auto bufc, auto maskc) {
    constexpr int BUF = decltype(bufc)::value;
    constexpr bool MASK = decltype(maskc)::value;
    auto& wcur = BUF ? wB : wA;
    auto& wnext = BUF ? wA : wB;
    const int64_t j0 = t * kBC;
    const bool more = t + 1 < ntiles;
    const int64_t jn = more ? j0 + kBC : j0;
    stK.load(tile_rsrc<D>(kh, jn, a.Sk));
    stV.load(tile_rsrc<D>(vh, jn, a.Sk));
    fetch_spd(jn, wnext);
    sched_fence();
    dq_tile<D, QB, MASK>(sK[BUF], sV[BUF], sT, off, qf, df, init_s, init_p, wcur, j0, a.Sk, sl2, acc);
    if (more) {
      stK.store(sK[BUF ^ 1]);
      stV.store(sV[BUF ^ 1]);
    }
    __syncthreads();
  };
  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  using Full = std::false_type;
  using Part = std::true_type;
  const int64_t nfull = FULL ? ntiles : a.Sk / kBC;
  int64_t t = 0;
  for (; t + 1 < nfull; t += 2) {
    step(t, B0(), Full());
    step(t + 1, B1(), Full());
  }
  if (t < nfull) {
    step(t, B0(), Full());
    if (!FULL && t + 1 < ntiles) step(t + 1, B1(), Part());
  } else if (!FULL && t < ntiles) {
    step(t, B0(), Part());
  }

#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int64_t i = qbase + qb * 32 + col;
    if (i >= a.Sq) continue;
    if (a.accumulate) {   // fp32 partial of the query shard, accumulated across ring steps
      float* dqa = reinterpret_cast<float*>(a.dq) + hq + i * D;
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int c = cb * 32 + 8 * u + 4 * g;
          float4 x = *reinterpret_cast<const float4*>(dqa + c);
          x.x += acc[qb][cb][4 * u] * a.scale; x.y += acc[qb][cb][4 * u + 1] * a.scale;
          x.z += acc[qb][cb][4 * u + 2] * a.scale; x.w += acc[qb][cb][4 * u + 3] * a.scale;
          *reinterpret_cast<float4*>(dqa + c) = x;
        }
      }
      continue;
    }
    uint16_t* dqp = reinterpret_cast<uint16_t*>(a.dq) + hq + i * D;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = cb * 32 + 8 * u + 4 * g;
        uint2 pk;
        pk.x = (uint32_t)f2bf(acc[qb][cb][4 * u] * a.scale) | ((uint32_t)f2bf(acc[qb][cb][4 * u + 1] * a.scale) << 16);
        pk.y = (uint32_t)f2bf(acc[qb][cb][4 * u + 2] * a.scale) | ((uint32_t)f2bf(acc[qb][cb][4 * u + 3] * a.scale) << 16);
        *reinterpret_cast<uint2*>(dqp + c) = pk;
      }
    }
  }
}

}  // namespace

hipError_t launch_dq_bf16(const BwdArgs& a, int d, hipStream_t s) {
  constexpr int QB = 1;
  constexpr int BR = kWaves * 32 * QB;
  const int64_t nqb = (a.Sq + BR - 1) / BR;
  const dim3 grid((unsigned)(nqb * a.H));
  const bool full = a.spd_vec && a.Sk % kBC == 0;
  if (d == 64) {
    if (full)
      hipLaunchKernelGGL((bwd_dq_bf16_kernel<64, QB, true, true>), grid, dim3(kThreads), 0, s, a);
    else if (a.spd_vec)
      hipLaunchKernelGGL((bwd_dq_bf16_kernel<64, QB, true, false>), grid, dim3(kThreads), 0, s, a);
    else
      hipLaunchKernelGGL((bwd_dq_bf16_kernel<64, QB, false, false>), grid, dim3(kThreads), 0, s, a);
  } else {
    if (full)
      hipLaunchKernelGGL((bwd_dq_bf16_kernel<32, QB, true, true>), grid, dim3(kThreads), 0, s, a);
    else if (a.spd_vec)
      hipLaunchKernelGGL((bwd_dq_bf16_kernel<32, QB, true, false>), grid, dim3(kThreads), 0, s, a);
    else
      hipLaunchKernelGGL((bwd_dq_bf16_kernel<32, QB, false, false>), grid, dim3(kThreads), 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace gt
