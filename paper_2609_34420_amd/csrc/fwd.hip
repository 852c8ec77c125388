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
// straight from registers. K and V tiles are staged row-major in LDS and
// shared by the 4 waves (V^T is read with transposing LDS reads); the
// per-head table (times log2 e) lives in LDS.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "stage.hpp"

namespace gt {

namespace {

constexpr int kWaves = 4;
constexpr int kThreads = kWaves * 64;
constexpr int kBC = 64;          // keys per LDS tile
constexpr float kRescaleSlack = 8.0f;   // log2 units the running max may lag

// Running softmax state of one 32-query block. Scores are kept relative to
// a reference max: the S^T accumulator starts at -msafe / (scale log2 e), so
// x = s * scale log2 e + bias is already x_abs - msafe and p = 2^x. The
// reference only moves (with a rescale of the accumulator) when a score
// passes it by more than the slack, which needs the one exchange between
// the lane halves; otherwise no cross-lane step is needed.
struct SoftmaxState {
  float m;        // reference max (log2 units), -inf before any finite score
  float l;        // this lane half's partial row sum, relative to m
  f32x16 init;    // -msafe / (scale log2 e), msafe = m or 0 while m = -inf
};

// Per-lane LDS element offsets of the operand reads (tile-relative; the
// 32-key block and 8-key step offsets are immediates).
template <int D>
struct FwdOffsets {
  int k[D / 16];          // K rows perm32(lane), feature chunk 2 kc + g
  int v[2][D / 32];       // transposing reads h = 0, 1 of V, feature block cb
  __device__ __forceinline__ FwdOffsets() {
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) k[kc] = row_operand_off<D>(kc);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int cb = 0; cb < D / 32; ++cb) v[h][cb] = tr_operand_off<D>(h, cb);
  }
};

// Both 32-key blocks' score products are issued before the first block's
// softmax, so the matrix cores work on block 1 while the vector ALUs work on
// block 0. A reference move in block 0 shifts the already computed block-1
// scores by the same amount.
template <int D, int QB, bool MASK>
__device__ __forceinline__ void fwd_tile(const uint16_t* sK, const uint16_t* sV, const float* sT,
                                         const FwdOffsets<D>& off,
                                         const bf16x8 (&qf)[QB][D / 16],
                                         const uint32_t (&w)[QB][kBC / 32][4], int64_t j0,
                                         int64_t Sk, float sl2, float inv_sl2,
                                         SoftmaxState (&st)[QB], f32x16 (&acc)[QB][D / 32]) {
  constexpr int KB = kBC / 32;
  constexpr int NKC = D / 16;
  constexpr int NCB = D / 32;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 5;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    f32x16 s[KB];
    float tb[KB][16];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) tb[kb][r] = sT[(w[qb][kb][r >> 2] >> (8 * (r & 3))) & 0xffu];
      s[kb] = st[qb].init;
#pragma unroll
      for (int kc = 0; kc < NKC; ++kc)
        s[kb] = mfma32(lds_b128(sK + kb * 32 * D + off.k[kc]), qf[qb][kc], s[kb]);
    }
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      float x[16];
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float xv = fmaf(s[kb][r], sl2, tb[kb][r]);
        if constexpr (MASK)
          x[r] = (j0 + kb * 32 + 16 * g + r < Sk) ? xv : -INFINITY;
        else
          x[r] = xv;
      }
      float mx = x[0];
#pragma unroll
      for (int r = 1; r < 16; ++r) mx = fmaxf(mx, x[r]);
      const float thr = (st[qb].m == -INFINITY) ? -INFINITY : kRescaleSlack;
      if (__any(mx > thr)) {
        // Move the reference: both halves agree on the new max.
        const float mall = fmaxf(mx, __shfl_xor(mx, 32));
        const float msafe_old = (st[qb].m == -INFINITY) ? 0.0f : st[qb].m;
        const float mnew = fmaxf(st[qb].m, mall + msafe_old);
        const float alpha = (mnew == -INFINITY) ? 1.0f : exp2_fast(st[qb].m - mnew);
        st[qb].l *= alpha;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
          for (int r = 0; r < 16; ++r) acc[qb][cb][r] *= alpha;
        const float msafe_new = (mnew == -INFINITY) ? 0.0f : mnew;
        const float shift = msafe_new - msafe_old;
#pragma unroll
        for (int r = 0; r < 16; ++r) x[r] -= shift;
        // later blocks of this tile were started from the old reference
        const float ds = shift * inv_sl2;
#pragma unroll
        for (int kb2 = kb + 1; kb2 < KB; ++kb2)
#pragma unroll
          for (int r = 0; r < 16; ++r) s[kb2][r] -= ds;
        st[qb].m = mnew;
        const float iv = -msafe_new * inv_sl2;
#pragma unroll
        for (int r = 0; r < 16; ++r) st[qb].init[r] = iv;
      }
      float ls = st[qb].l;
#pragma unroll
      for (int q = 0; q < 2; ++q) {
        float p[8];
#pragma unroll
        for (int r = 0; r < 8; ++r) p[r] = exp2_fast(x[8 * q + r]);
        const bf16x8 pb = cvt_bf16x8(p);
        ls = sum_bf16x8(pb, ls);       // the row sum of exactly the P that P V uses
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
          const uint16_t* vt = sV + (kb * 32 + 8 * q) * D;
          acc[qb][cb] = mfma32(lds_tr_operand(vt, off.v[0][cb], off.v[1][cb]), pb, acc[qb][cb]);
        }
      }
      st[qb].l = ls;
    }
  }
}

// VEC: spd rows are 16-byte aligned. FULL: VEC and Sk a multiple of the key
// tile, so every spd group is loaded whole and no tile needs masking.
template <int D, int QB, bool OUT_F32, bool VEC, bool FULL>
__global__ __launch_bounds__(kThreads, 2) void fwd_bf16_kernel(FwdArgs a) {
  constexpr int KB = kBC / 32;
  constexpr int NKC = D / 16;
  constexpr int NCB = D / 32;
  constexpr int BR = kWaves * 32 * QB;
  using Dma = TileDma<D, kWaves>;     // K and V
  static_assert(kBC == kTileRows, "key tile is one staged tile");

  // Three-stage ring of K / V tiles, one array per stage so that no read of
  // one stage can be taken to alias the copy into another.
  __shared__ __attribute__((aligned(16))) uint16_t sK0[kBC * D], sK1[kBC * D], sK2[kBC * D];
  __shared__ __attribute__((aligned(16))) uint16_t sV0[kBC * D], sV1[kBC * D], sV2[kBC * D];
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

  const uint16_t* qh = reinterpret_cast<const uint16_t*>(a.q) + (int64_t)h * a.Sq * D;
  const uint16_t* kh = reinterpret_cast<const uint16_t*>(a.k) + (int64_t)h * a.Sk * D;
  const uint16_t* vh = reinterpret_cast<const uint16_t*>(a.v) + (int64_t)h * a.Sk * D;
  const float sl2 = a.scale * kLog2e;

  // Q^T operands; rows past Sq load the clamped row Sq-1 (their output is
  // not stored).
  bf16x8 qf[QB][NKC];
  int64_t qrow[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int64_t i = qbase + qb * 32 + col;
    qrow[qb] = i < a.Sq ? i : a.Sq - 1;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc)
      qf[qb][kc] = *reinterpret_cast<const bf16x8*>(qh + qrow[qb] * D + kc * 16 + g * 8);
  }

  // spd bytes of key group j..j+15 of the lane's query row: one 16-byte raw
  // buffer load (scalar base per wave, lane offset row*ld + 16 g, scalar key
  // offset), or byte loads for the partial last tile and unaligned slices.
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

  const float inv_sl2 = 1.0f / sl2;
  SoftmaxState sm[QB];
  f32x16 acc[QB][NCB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    sm[qb].m = -INFINITY;
    sm[qb].l = 0.0f;
    sm[qb].init = zero_f32x16();
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[qb][cb] = zero_f32x16();
  }

  const int64_t ntiles = (a.Sk + kBC - 1) / kBC;
  const FwdOffsets<D> off;
  const Dma dma(wave);
  uint32_t w0[QB][KB][4], w1[QB][KB][4], w2[QB][KB][4];   // spd words, by tile % 3

  // Copy tile t (clamped to the last tile) into stage s and fetch its spd
  // words: Dma::NLOADS + SPD_LOADS vector-memory ops per wave.
  constexpr int SPD_LOADS = QB * KB;
#define GT_FWD_ISSUE(t_, S_)                                                                    \
  {                                                                                            \
    const int64_t j_ = ((t_) < ntiles ? (t_) : ntiles - 1) * kBC;                              \
    dma.load(tile_rsrc<D>(kh, j_, a.Sk), tile_rsrc<D>(vh, j_, a.Sk),                          \
             (S_) == 0 ? sK0 : ((S_) == 1 ? sK1 : sK2), (S_) == 0 ? sV0 : ((S_) == 1 ? sV1 : sV2)); \
    fetch_spd(j_, (S_) == 0 ? w0 : ((S_) == 1 ? w1 : w2));                                    \
  }
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2>;
  if (ntiles > 0) {
    GT_FWD_ISSUE(0, 0)
    GT_FWD_ISSUE(1, 1)
  }
  __syncthreads();     // table, and the copy of tile 0 (waits for every load)

  // Tile t from stage S = t % 3: copy tile t + 2 into stage (S + 2) % 3
  // (last read in step t - 1, before that step's barrier), compute, then
  // wait until this wave's copy of tile t + 1 has landed (only the spd
  // words of tile t + 1 and this step's loads may still be in flight) and
  // meet the other waves at the barrier.
  auto step = [&](int64_t t, auto stagec, auto maskc) {
    constexpr int S = decltype(stagec)::value;
    constexpr bool MASK = decltype(maskc)::value;
    GT_FWD_ISSUE(t + 2, (S + 2) % 3)
    sched_fence();
    auto& w = S == 0 ? w0 : (S == 1 ? w1 : w2);
    const uint16_t* k_s = S == 0 ? sK0 : (S == 1 ? sK1 : sK2);
    const uint16_t* v_s = S == 0 ? sV0 : (S == 1 ? sV1 : sV2);
    fwd_tile<D, QB, MASK>(k_s, v_s, sT, off, qf, w, t * kBC, a.Sk, sl2, inv_sl2, sm, acc);
    if constexpr (FULL)
      wait_vmcnt<2 * SPD_LOADS + Dma::NLOADS>();
    else
      wait_vmcnt<0>();     // the unaligned spd path issues a variable number of loads
    __builtin_amdgcn_s_barrier();
  };
  using Full = std::false_type;     // every key of the tile exists
  using Part = std::true_type;      // keys past Sk masked
  const int64_t nfull = FULL ? ntiles : a.Sk / kBC;
  int64_t t = 0;
  for (; t + 3 <= nfull; t += 3) {
    step(t, S0(), Full());
    step(t + 1, S1(), Full());
    step(t + 2, S2(), Full());
  }
  // At most two full tiles and the partial one remain, in stages 0, 1, 2.
  if constexpr (FULL) {
    if (t < ntiles) step(t, S0(), Full());
    if (t + 1 < ntiles) step(t + 1, S1(), Full());
  } else {
    if (t < ntiles) step(t, S0(), Part());
    if (t + 1 < ntiles) step(t + 1, S1(), Part());
    if (t + 2 < ntiles) step(t + 2, S2(), Part());
  }

  // Epilogue: O = O_acc / l, LSE = (m + log2 l) ln 2.
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float lt = sm[qb].l + __shfl_xor(sm[qb].l, 32);
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
      a.lse[(int64_t)h * a.Sq + i] = lt > 0.0f ? (sm[qb].m + __log2f(lt)) * kLn2 : -INFINITY;
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
  const dim3 grid((unsigned)(nqb * a.H));
  if (a.spd_vec && a.Sk % kBC == 0)
    hipLaunchKernelGGL((fwd_bf16_kernel<D, QB, OUT_F32, true, true>), grid, dim3(kThreads), 0, s, a);
  else if (a.spd_vec)
    hipLaunchKernelGGL((fwd_bf16_kernel<D, QB, OUT_F32, true, false>), grid, dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((fwd_bf16_kernel<D, QB, OUT_F32, false, false>), grid, dim3(kThreads), 0, s, a);
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
    return out_f32 ? launch_fwd_bf16<32, 2, true>(a, s) : launch_fwd_bf16<32, 2, false>(a, s);
  }
  return d == 64 ? launch_fwd_f32<64>(a, s) : launch_fwd_f32<32>(a, s);
}

}  // namespace gt
