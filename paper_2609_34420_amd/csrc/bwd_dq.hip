// Backward, query-stationary stage: dQ (bf16).
//
// Same layout as the forward: each wave owns 32 queries, computes
// S^T = K Q^T and dP^T = V dO^T with the queries on the lanes, forms
// dS^T = P^T * (dP^T - Dlt) from the saved log-sum-exp, and accumulates
// dQ^T += K^T dS^T with dS^T straight from registers (K^T by transposing LDS
// reads). K and V tiles stream through a three-stage LDS ring filled by
// direct buffer -> LDS loads.
//
// Per score element the vector work is one FMA, one exp2, one multiply and
// half a bf16 conversion:
//   * the score accumulator starts from the bias table entries (kept in LDS
//     as bias / scale, one copy per lane), so the matrix cores produce
//     bias / scale + q.k, and x = that * scale log2(e) - LSE log2(e) with the
//     lane's (the query's) LSE as the FMA addend;
//   * -Dlt enters dP through one more matrix product: a ones column of the
//     key operand against the query's -Dlt split into three bf16 terms
//     (exact to about 2^-25 of Dlt), with the accumulator started at zero.
// The score and dP products of the next 32-key block are issued before the
// current block's element work, so the matrix cores overlap it.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "stage.hpp"

namespace gt {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kBC = 64;            // keys per LDS tile
constexpr int kKB = kBC / 32;      // 32-key blocks per tile

// Per-lane LDS element offsets of the operand reads (tile-relative; 32-key
// block and 8-key step offsets are immediates). K and V rows share one
// pattern.
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

// The wave's stationary operands and statistics.
template <int D>
struct DqLane {
  bf16x8 qf[D / 16];      // Q^T
  bf16x8 df[D / 16];      // dO^T
  bf16x8 ones;            // key operand of the -Dlt product: 1 at k = 0, 1, 2
  bf16x8 dlt;             // query operand: -Dlt as three bf16 terms at k = 0, 1, 2
  float mlse2;            // -LSE log2 e; -inf for padded or empty rows (P = 0)
};

// Score and dP products of one 32-key block (key block kb of a staged tile)
// over the NK 16-feature chunks that hold data.
template <int D, int NK>
__device__ __forceinline__ void issue_block(const float* tab, const uint32_t (&w)[4], uint32_t lane4,
                                            const uint16_t* sK, const uint16_t* sV,
                                            const DqOffsets<D>& off, int kb, const DqLane<D>& ln,
                                            f32x16& s, f32x16& dp) {
  load_bias(tab, w, lane4, s);
  dp = mfma32(ln.ones, ln.dlt, zero_f32x16());
#pragma unroll
  for (int kc = 0; kc < NK; ++kc) {
    s = mfma32(lds_b128(sK + kb * 32 * D + off.row[kc]), ln.qf[kc], s);
    dp = mfma32(lds_b128(sV + kb * 32 * D + off.row[kc]), ln.df[kc], dp);
  }
}

template <int D>
__device__ __forceinline__ void read_kt(const uint16_t* sK, const DqOffsets<D>& off, int kb,
                                        bf16x8 (&kt)[2][D / 32]) {
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int cb = 0; cb < D / 32; ++cb)
      kt[q][cb] = lds_tr_operand(sK + (kb * 32 + 8 * q) * D, off.kt[0][cb], off.kt[1][cb]);
}

// dS^T of one block and dQ^T += K^T dS^T. MASK: keys at or past jrem (relative
// to the block) are padding.
template <int D, bool MASK>
__device__ __forceinline__ void block_dq(const f32x16& s, const f32x16& dp, const bf16x8 (&kt)[2][D / 32],
                                         int64_t jrem, float sl2, float mlse2, f32x16 (&acc)[D / 32]) {
  const int g = (threadIdx.x >> 5) & 1;
  float ds[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    float pv = exp2_fast(fmaf(s[r], sl2, mlse2));
    if constexpr (MASK) pv = (16 * g + r < jrem) ? pv : 0.0f;
    ds[r] = pv * dp[r];
  }
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const bf16x8 db = cvt_bf16x8(ds + 8 * q);
#pragma unroll
    for (int cb = 0; cb < D / 32; ++cb) acc[cb] = mfma32(kt[q][cb], db, acc[cb]);
  }
}

// D: the tile's head dim (32 or 64); DS <= D: the head dim of the tensors
// (8 and 16 run on 32-wide tiles whose extra features are zero). VEC: spd
// rows are 16-byte aligned. FULL: VEC and Sk a multiple of the key tile, so
// every spd group is loaded whole and no tile needs masking.
template <int D, int DS, bool VEC, bool FULL>
__global__ __launch_bounds__(kThreads, 1) void bwd_dq_bf16_kernel(BwdArgs a) {
  constexpr int NKC = D / 16;
  constexpr int NKS = (DS + 15) / 16;   // feature chunks that hold data
  constexpr int NCB = D / 32;
  constexpr int BR = kWaves * 32;
  using Dma = TileDma<D, kWaves, DS>;     // K and V
  static_assert(kBC == kTileRows, "key tile is one staged tile");

  __shared__ __attribute__((aligned(16))) uint16_t sK0[kBC * D], sK1[kBC * D], sK2[kBC * D];
  __shared__ __attribute__((aligned(16))) uint16_t sV0[kBC * D], sV1[kBC * D], sV2[kBC * D];
  __shared__ __attribute__((aligned(16))) float sTab[kLaneTableFloats];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = wave_id();
  const int col = lane & 31, g = lane >> 5;
  const uint32_t lane4 = (uint32_t)lane * 4u;

  const int64_t nqb = (a.Sq + BR - 1) / BR;
  const int64_t lid = xcd_remap(blockIdx.x, nqb * a.H);
  const int h = (int)(lid % a.H);
  const int64_t qblk = lid / a.H;
  const int64_t qbase = qblk * BR + (int64_t)wave * 32;

  fill_lane_table(sTab, a.table + (int64_t)table_row(a, h) * a.n_buckets, a.n_buckets, a.scale, kThreads);

  const int64_t hq = (int64_t)h * a.Sq * DS;   // query-side rows
  const int64_t hk = (int64_t)h * a.Sk * DS;   // key-side rows
  const uint16_t* qh = reinterpret_cast<const uint16_t*>(a.q) + hq;
  const uint16_t* kh = reinterpret_cast<const uint16_t*>(a.k) + hk;
  const uint16_t* vh = reinterpret_cast<const uint16_t*>(a.v) + hk;
  const uint16_t* oh = reinterpret_cast<const uint16_t*>(a.d_o) + hq;
  const float sl2 = a.scale * kLog2e;

  // Stationary operands; rows past Sq load the clamped row Sq-1 and get
  // P = 0; their dQ is not stored.
  DqLane<D> ln;
  const int64_t i = qbase + col;
  const int64_t qrow = i < a.Sq ? i : a.Sq - 1;
#pragma unroll
  for (int kc = 0; kc < NKC; ++kc) {
    const bool in = DS == D || kc * 16 + g * 8 < DS;
    ln.qf[kc] = in ? *reinterpret_cast<const bf16x8*>(qh + qrow * DS + kc * 16 + g * 8) : zero_bf16x8();
    ln.df[kc] = in ? *reinterpret_cast<const bf16x8*>(oh + qrow * DS + kc * 16 + g * 8) : zero_bf16x8();
  }
  {
    const float l2 = a.lse2[(int64_t)h * a.Sq + qrow];
    const float dl = i < a.Sq ? a.dlt[(int64_t)h * a.Sq + qrow] : 0.0f;
    ln.mlse2 = i < a.Sq ? -l2 : -INFINITY;
    const __bf16 t0 = (__bf16)(-dl);
    const float r1 = -dl - (float)t0;
    const __bf16 t1 = (__bf16)r1;
    const __bf16 t2 = (__bf16)(r1 - (float)t1);
    const __bf16 z = (__bf16)0.0f, one = (__bf16)1.0f;
    ln.dlt = zero_bf16x8();
    ln.ones = zero_bf16x8();
    if (g == 0) {
      ln.dlt[0] = t0; ln.dlt[1] = t1; ln.dlt[2] = t2;
      ln.ones[0] = one; ln.ones[1] = one; ln.ones[2] = one;
    }
    (void)z;
  }
  f32x16 acc[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) acc[cb] = zero_f32x16();

  // spd bytes of key group j..j+15 of the lane's query row: one 16-byte raw
  // buffer load, or byte loads for the partial last tile and unaligned
  // slices.
  const int64_t ld = a.ld_spd;
  const int64_t rb = qbase < a.Sq ? qbase : a.Sq - 1;
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(seq_spd(a, h) + (a.row_off + rb) * ld + a.col_off);
  const uint32_t voff = (uint32_t)((qrow - rb) * ld) + 16u * g;
  const int64_t ntiles = (a.Sk + kBC - 1) / kBC;
  auto fetch_spd = [&](int64_t tt, uint32_t (&w)[kKB][4]) {
    const int64_t jt = (tt < ntiles ? tt : ntiles - 1) * kBC;
    if (FULL || (VEC && jt + kBC <= a.Sk)) {
#pragma unroll
      for (int kb = 0; kb < kKB; ++kb) buf_u128(rs, voff, (uint32_t)(jt + kb * 32), w[kb]);
    } else {
      const uint8_t* row = seq_spd(a, h) + (a.row_off + qrow) * ld + a.col_off;
#pragma unroll
      for (int kb = 0; kb < kKB; ++kb) load_spd16_bytes(row, jt + kb * 32 + 16 * g, a.Sk, w[kb]);
    }
  };

  const DqOffsets<D> off;
  const Dma dma(wave);
  constexpr int SPD_LOADS = kKB;
#define GT_DQ_STAGE(S_, K_, V_)                                                                 \
  uint16_t* K_ = (S_) == 0 ? sK0 : ((S_) == 1 ? sK1 : sK2);                                   \
  uint16_t* V_ = (S_) == 0 ? sV0 : ((S_) == 1 ? sV1 : sV2);
  auto copy_tile = [&](int64_t tt, auto stagec) {
    constexpr int S = decltype(stagec)::value;
    GT_DQ_STAGE(S, k_s, v_s)
    const int64_t j_ = (tt < ntiles ? tt : ntiles - 1) * kBC;
    dma.load(tile_rsrc<DS>(kh, j_, a.Sk), tile_rsrc<DS>(vh, j_, a.Sk), k_s, v_s);
  };
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2>;

  if constexpr (FULL) {
    // K/V tile t in stage t % 3 (copied two tiles ahead); spd words of tile
    // t in register set t % 2 (fetched one tile ahead).
    uint32_t wA[kKB][4], wB[kKB][4];
    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;
    f32x16 s0, dp0;     // products of the current tile's first key block
    if (ntiles > 0) {
      copy_tile(0, S0());
      copy_tile(1, S1());
      copy_tile(2, S2());
      fetch_spd(0, wA);
      fetch_spd(1, wB);
      wait_vmcnt<0>();
      __syncthreads();     // table, tiles 0..2
      issue_block<D, NKS>(sTab, wA[0], lane4, sK0, sV0, off, 0, ln, s0, dp0);
    }
    // Tile t: products of key block 1 issued, then block 0's element work
    // and dQ product; block 1's K^T operands read; spd words of tile t + 2
    // fetched into the freed set; tile boundary (tile t + 1 landed, barrier,
    // stage refilled with tile t + 3); tile t + 1's block-0 products issued;
    // block 1's element work and dQ product.
    auto step = [&](int64_t t, auto stagec, auto setc) {
      constexpr int S = decltype(stagec)::value;
      constexpr int SN = (S + 1) % 3;
      constexpr int P = decltype(setc)::value;
      GT_DQ_STAGE(S, k_s, v_s)
      GT_DQ_STAGE(SN, k_n, v_n)
      auto& w = P == 0 ? wA : wB;
      auto& w_n = P == 0 ? wB : wA;
      f32x16 s1, dp1;
      bf16x8 kt[2][NCB];
      issue_block<D, NKS>(sTab, w[1], lane4, k_s, v_s, off, 1, ln, s1, dp1);
      read_kt<D>(k_s, off, 0, kt);
      block_dq<D, false>(s0, dp0, kt, kBC, sl2, ln.mlse2, acc);
      read_kt<D>(k_s, off, 1, kt);
      fetch_spd(t + 2, w);
      sched_fence();
      wait_vmcnt<SPD_LOADS + Dma::NLOADS>();
      __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): this wave's reads of stage S done
      __builtin_amdgcn_s_barrier();
      copy_tile(t + 3, stagec);
      sched_fence();
      issue_block<D, NKS>(sTab, w_n[0], lane4, k_n, v_n, off, 0, ln, s0, dp0);
      block_dq<D, false>(s1, dp1, kt, kBC, sl2, ln.mlse2, acc);
    };
    int64_t t = 0;
    for (; t + 6 <= ntiles; t += 6) {
      step(t, S0(), P0());
      step(t + 1, S1(), P1());
      step(t + 2, S2(), P0());
      step(t + 3, S0(), P1());
      step(t + 4, S1(), P0());
      step(t + 5, S2(), P1());
    }
    if (t < ntiles) step(t, S0(), P0());
    if (t + 1 < ntiles) step(t + 1, S1(), P1());
    if (t + 2 < ntiles) step(t + 2, S2(), P0());
    if (t + 3 < ntiles) step(t + 3, S0(), P1());
    if (t + 4 < ntiles) step(t + 4, S1(), P0());
  } else {
    // Ragged or unaligned: spd words fetched two tiles ahead in three sets,
    // one tile per step, every wait drains the loads.
    uint32_t w0[kKB][4], w1[kKB][4], w2[kKB][4];
    if (ntiles > 0) {
      copy_tile(0, S0());
      fetch_spd(0, w0);
      copy_tile(1, S1());
      fetch_spd(1, w1);
    }
    wait_vmcnt<0>();
    __syncthreads();     // table, and the copy of tile 0
    auto step = [&](int64_t t, auto stagec, auto maskc) {
      constexpr int S = decltype(stagec)::value;
      constexpr bool MASK = decltype(maskc)::value;
      GT_DQ_STAGE(S, k_s, v_s)
      copy_tile(t + 2, std::integral_constant<int, (S + 2) % 3>());
      fetch_spd(t + 2, S == 0 ? w2 : (S == 1 ? w0 : w1));
      sched_fence();
      auto& w = S == 0 ? w0 : (S == 1 ? w1 : w2);
      const int64_t jrem = a.Sk - t * kBC;
#pragma unroll
      for (int kb = 0; kb < kKB; ++kb) {
        f32x16 s, dp;
        bf16x8 kt[2][NCB];
        issue_block<D, NKS>(sTab, w[kb], lane4, k_s, v_s, off, kb, ln, s, dp);
        read_kt<D>(k_s, off, kb, kt);
        block_dq<D, MASK>(s, dp, kt, jrem - kb * 32, sl2, ln.mlse2, acc);
      }
      wait_vmcnt<0>();
      __builtin_amdgcn_s_barrier();
    };
    using Full = std::false_type;
    using Part = std::true_type;
    const int64_t nfull = a.Sk / kBC;
    int64_t t = 0;
    for (; t + 3 <= nfull; t += 3) {
      step(t, S0(), Full());
      step(t + 1, S1(), Full());
      step(t + 2, S2(), Full());
    }
    if (t < ntiles) step(t, S0(), Part());
    if (t + 1 < ntiles) step(t + 1, S1(), Part());
    if (t + 2 < ntiles) step(t + 2, S2(), Part());
  }
  wait_vmcnt<0>();     // drain the clamped copies issued past the last tile
#undef GT_DQ_STAGE

  if (i >= a.Sq) return;
  if (a.accumulate) {   // fp32 partial of the query shard, accumulated across ring steps
    float* dqa = reinterpret_cast<float*>(a.dq) + hq + i * DS;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = cb * 32 + 8 * u + 4 * g;
        if (c >= DS) continue;               // zero padding of a narrow head dim
        float4 x = *reinterpret_cast<const float4*>(dqa + c);
        x.x += acc[cb][4 * u] * a.scale; x.y += acc[cb][4 * u + 1] * a.scale;
        x.z += acc[cb][4 * u + 2] * a.scale; x.w += acc[cb][4 * u + 3] * a.scale;
        *reinterpret_cast<float4*>(dqa + c) = x;
      }
    }
    return;
  }
  uint16_t* dqp = reinterpret_cast<uint16_t*>(a.dq) + hq + i * DS;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = cb * 32 + 8 * u + 4 * g;
      if (c >= DS) continue;
      uint2 pk;
      pk.x = (uint32_t)f2bf(acc[cb][4 * u] * a.scale) | ((uint32_t)f2bf(acc[cb][4 * u + 1] * a.scale) << 16);
      pk.y = (uint32_t)f2bf(acc[cb][4 * u + 2] * a.scale) | ((uint32_t)f2bf(acc[cb][4 * u + 3] * a.scale) << 16);
      *reinterpret_cast<uint2*>(dqp + c) = pk;
    }
  }
}

template <int D, int DS>
void launch_dq_t(const BwdArgs& a, hipStream_t s) {
  constexpr int BR = kWaves * 32;
  const int64_t nqb = (a.Sq + BR - 1) / BR;
  const dim3 grid((unsigned)(nqb * a.H));
  if (a.spd_vec && a.Sk % kBC == 0)
    hipLaunchKernelGGL((bwd_dq_bf16_kernel<D, DS, true, true>), grid, dim3(kThreads), 0, s, a);
  else if (a.spd_vec)
    hipLaunchKernelGGL((bwd_dq_bf16_kernel<D, DS, true, false>), grid, dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((bwd_dq_bf16_kernel<D, DS, false, false>), grid, dim3(kThreads), 0, s, a);
}

}  // namespace

hipError_t launch_dq_bf16(const BwdArgs& a, int d, hipStream_t s) {
  switch (d) {
    case 8: launch_dq_t<32, 8>(a, s); break;
    case 16: launch_dq_t<32, 16>(a, s); break;
    case 32: launch_dq_t<32, 32>(a, s); break;
    default: launch_dq_t<64, 64>(a, s); break;
  }
  return hipGetLastError();
}

}  // namespace gt
