// Forward / ring-step kernels: blockwise biased attention with online softmax.
//
// S = scale * Q K^T + table[h, spd[row_off + i, col_off + j]]   (Eq. (1); Eq. (2)
// for a ring step), softmax statistics updated block by block with the bias
// already inside the scores (Section III-A-1 part 3).
//
// bf16 path (gfx950 matrix cores). Each wave owns 64 queries (two 32-query
// blocks) and computes the TRANSPOSED score tiles S^T = K Q^T, so every lane
// owns one query (lane & 31) and 16 consecutive keys per 32-key block: the
// row sum is lane-local plus one exchange between the lane halves at the
// end, and the lane's 16 spd bytes are one 16-byte load. P^T then feeds
// O^T += V^T P^T straight from registers. K and V tiles are staged row-major
// in LDS and shared by the 8 waves; each operand read serves both query
// blocks of a wave (V^T through transposing LDS reads).
//
// The bias enters as the starting value of the score accumulator: the table
// is kept in LDS as bias / scale, so the matrix cores produce
// bias / scale + q.k and one FMA per element gives the base-2 exponent
// (q.k scale + bias) log2(e) - m. The table has one copy per lane (entry
// (b, lane) at byte 256 b + 4 lane): a single byte permute turns a spd byte
// into the lane's entry address, every byte value 0..255 has an entry (0 past
// n_buckets), and the reads are free of bank conflicts.
//
// Softmax reference: the reference max m of a row only moves when needed.
// The bf16 row sum of each 16-key half block is computed anyway (it is the
// sum of exactly the P that P V uses); while it stays at or below 256 every
// p of the block is at most 256 and the block is accepted as is. Otherwise
// (or while a row has no finite score yet) the wave takes the exact path:
// the block max moves the reference, the accumulator and sum are rescaled
// and the block is recomputed. Accepted blocks therefore never hold p > 256,
// and the reference is always a score the row attained, so the final sum is
// at least 1 and nothing that matters underflows.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "stage.hpp"
#include "fwd_tile.hpp"

namespace gt {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kBC = 64;            // keys per LDS tile
constexpr int kQB = 2;             // 32-query blocks per wave
constexpr int kKB = kBC / 32;      // 32-key blocks per tile
// Unpipelined tile (ragged or unaligned shapes): for each 32-key block the
// score products of both query blocks, then their softmax and P V.
template <int D, int NK, bool MASK>
__device__ __forceinline__ void fwd_tile(const uint16_t* sK, const uint16_t* sV, const float* tab,
                                         const FwdOffsets<D>& off,
                                         const bf16x8 (&qf)[kQB][D / 16],
                                         const uint32_t (&w)[kQB][kKB][4], uint32_t lane4,
                                         int64_t jrem, float sl2, SoftmaxState (&st)[kQB],
                                         f32x16 (&acc)[kQB][D / 32]) {
  constexpr int NCB = D / 32;
#pragma unroll
  for (int kb = 0; kb < kKB; ++kb) {
    f32x16 s[kQB];
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb) issue_scores<D, NK>(tab, w[qb][kb], lane4, sK, off.k, kb, qf[qb], s[qb]);
    bf16x8 vop[2][NCB];
    read_v<D>(sV, off, kb, vop);
#pragma unroll
    for (int qb = 0; qb < kQB; ++qb)
      softmax_pv<D, MASK>(s[qb], vop, jrem - kb * 32, sl2, st[qb], acc[qb]);
  }
}

// D: the tile's head dim (32 or 64); DS <= D: the head dim of the tensors
// (8 and 16 run on 32-wide tiles whose extra features are zero). VEC: spd
// rows are 16-byte aligned. FULL: VEC and Sk a multiple of the key tile, so
// every spd group is loaded whole and no tile needs masking. SKIP: Sq is not
// a multiple of the workgroup's rows, so some waves may own no row. PAIR
// (batches of sequences of at most 256 nodes): the two halves of the
// workgroup (waves 0-3 and 4-7) take the same head of two consecutive
// sequences, which share the bias table; each half stages its own K/V.
template <int D, int DS, bool OUT_F32, bool VEC, bool FULL, bool SKIP, bool PAIR = false>
__global__ __launch_bounds__(kThreads, 1) void fwd_bf16_kernel(FwdArgs a) {
  constexpr int NKC = D / 16;
  constexpr int NKS = (DS + 15) / 16;   // feature chunks that hold data
  constexpr int NCB = D / 32;
  constexpr int NWI = PAIR ? kWaves / 2 : kWaves;   // waves per sequence
  constexpr int BR = NWI * 32 * kQB;
  using Dma = TileDma<D, NWI, DS>;        // K and V
  static_assert(kBC == kTileRows, "key tile is one staged tile");

  // Three-stage ring of K / V tiles, one array per stage so that no read of
  // one stage can be taken to alias the copy into another; the bias table,
  // one copy per lane: entry (b, lane) at float index 64 b + lane.
  constexpr int NI = PAIR ? 2 : 1;
  __shared__ __attribute__((aligned(16))) uint16_t sK0[NI * kBC * D], sK1[NI * kBC * D], sK2[NI * kBC * D];
  __shared__ __attribute__((aligned(16))) uint16_t sV0[NI * kBC * D], sV1[NI * kBC * D], sV2[NI * kBC * D];
  __shared__ __attribute__((aligned(16))) float sTab[kLaneTableFloats];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave_all = wave_id();
  const int item = PAIR ? wave_all / NWI : 0;        // the workgroup half (sequence) of the wave
  const int wave = PAIR ? wave_all % NWI : wave_all;
  const int col = lane & 31, g = lane >> 5;
  const uint32_t lane4 = (uint32_t)lane * 4u;

  const int64_t nqb = (a.Sq + BR - 1) / BR;
  int h;
  int64_t qblk;
  bool item_ok = true;
  if constexpr (PAIR) {
    // workgroup = (sequence pair, head); Sq <= BR, so one row block
    const int nseq = a.H / a.hpb;
    const int64_t lid = xcd_remap(blockIdx.x, (int64_t)((nseq + 1) / 2) * a.hpb);
    const int hh = (int)(lid % a.hpb);
    const int seq = (int)(lid / a.hpb) * 2 + item;
    item_ok = seq < nseq;
    h = (item_ok ? seq : seq - 1) * a.hpb + hh;
    qblk = 0;
  } else {
    const int64_t lid = xcd_remap(blockIdx.x, nqb * a.H);
    h = (int)(lid % a.H);
    qblk = lid / a.H;
  }
  const int64_t qbase = qblk * BR + (int64_t)wave * 32 * kQB;
  // A wave whose rows all lie past Sq (short sequences) still takes its
  // share of the tile copies, spd loads, waits and barriers, but skips the
  // products and the softmax, leaving its SIMD to the other wave.
  const bool active = (!SKIP || qbase < a.Sq) && item_ok;
  const int item_off = item * kBC * D;               // this half's K/V staging

  fill_lane_table(sTab, a.table + (int64_t)table_row(a, h) * a.n_buckets, a.n_buckets, a.scale, kThreads);

  const uint16_t* qh = reinterpret_cast<const uint16_t*>(a.q) + (int64_t)h * a.Sq * DS;
  const uint16_t* kh = reinterpret_cast<const uint16_t*>(a.k) + (int64_t)h * a.Sk * DS;
  const uint16_t* vh = reinterpret_cast<const uint16_t*>(a.v) + (int64_t)h * a.Sk * DS;
  const float sl2 = a.scale * kLog2e;

  // Q^T operands; rows past Sq load the clamped row Sq-1 (their output is
  // not stored).
  bf16x8 qf[kQB][NKC];
  int64_t qrow[kQB];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
    const int64_t i = qbase + qb * 32 + col;
    qrow[qb] = i < a.Sq ? i : a.Sq - 1;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) {
      if (DS == D || kc * 16 + g * 8 < DS)
        qf[qb][kc] = *reinterpret_cast<const bf16x8*>(qh + qrow[qb] * DS + kc * 16 + g * 8);
      else
        qf[qb][kc] = zero_bf16x8();
    }
  }

  // spd bytes of key group j..j+15 of the lane's query row: one 16-byte raw
  // buffer load (scalar base per wave, lane offset row*ld + 16 g, scalar key
  // offset), or byte loads for the partial last tile and unaligned slices.
  const int64_t ld = a.ld_spd;
  const int64_t rb = qbase < a.Sq ? qbase : a.Sq - 1;
  const __amdgpu_buffer_rsrc_t rs = make_rsrc(seq_spd(a, h) + (a.row_off + rb) * ld + a.col_off);
  uint32_t voff[kQB];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) voff[qb] = (uint32_t)((qrow[qb] - rb) * ld) + 16u * g;
  auto fetch_spd = [&](int64_t jt, uint32_t (&w)[kQB][kKB][4]) {
    if (FULL || (VEC && jt + kBC <= a.Sk)) {
#pragma unroll
      for (int qb = 0; qb < kQB; ++qb)
#pragma unroll
        for (int kb = 0; kb < kKB; ++kb) buf_u128(rs, voff[qb], (uint32_t)(jt + kb * 32), w[qb][kb]);
    } else {
#pragma unroll
      for (int qb = 0; qb < kQB; ++qb) {
        const uint8_t* row = seq_spd(a, h) + (a.row_off + qrow[qb]) * ld + a.col_off;
#pragma unroll
        for (int kb = 0; kb < kKB; ++kb) load_spd16_bytes(row, jt + kb * 32 + 16 * g, a.Sk, w[qb][kb]);
      }
    }
  };

  SoftmaxState sm[kQB];
  f32x16 acc[kQB][NCB];
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
    sm[qb].m = -INFINITY;
    sm[qb].mneg = 0.0f;
    sm[qb].l = 0.0f;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[qb][cb] = zero_f32x16();
  }

  const int64_t ntiles = (a.Sk + kBC - 1) / kBC;
  const FwdOffsets<D> off;
  const Dma dma(wave);
  constexpr int SPD_LOADS = kQB * kKB;
#define GT_FWD_STAGE(S_, K_, V_)                                                                \
  uint16_t* K_ = ((S_) == 0 ? sK0 : ((S_) == 1 ? sK1 : sK2)) + item_off;                      \
  uint16_t* V_ = ((S_) == 0 ? sV0 : ((S_) == 1 ? sV1 : sV2)) + item_off;
  // K/V tiles: a three-stage LDS ring, tile t in stage t % 3, copied two
  // tiles ahead (Dma::NLOADS vector-memory ops per wave); tiles past the
  // end are clamped to the last one.
  auto copy_tile = [&](int64_t tt, auto stagec) {
    constexpr int S = decltype(stagec)::value;
    GT_FWD_STAGE(S, k_s, v_s)
    const int64_t j_ = (tt < ntiles ? tt : ntiles - 1) * kBC;
    dma.load(tile_rsrc<DS>(kh, j_, a.Sk), tile_rsrc<DS>(vh, j_, a.Sk), k_s, v_s);
  };
  auto spd_of = [&](int64_t tt, uint32_t (&w)[kQB][kKB][4]) {
    fetch_spd((tt < ntiles ? tt : ntiles - 1) * kBC, w);
  };
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2>;

  if constexpr (FULL) {
    // spd words: two register sets, tile t in set t % 2, fetched one tile
    // ahead (SPD_LOADS vector-memory ops per wave).
    uint32_t wA[kQB][kKB][4], wB[kQB][kKB][4];
    using P0 = std::integral_constant<int, 0>;
    using P1 = std::integral_constant<int, 1>;
    f32x16 s0;        // score accumulator of the current tile's first unit
    if (ntiles > 0) {
      copy_tile(0, S0());
      copy_tile(1, S1());
      copy_tile(2, S2());
      spd_of(0, wA);
      spd_of(1, wB);
      wait_vmcnt<0>();
      __syncthreads();     // table, and tiles 0..2
      if (active) issue_scores<D, NKS>(sTab, wA[0][0], lane4, sK0 + item_off, off.k, 0, qf[0], s0);
    }
    // Tile t from stage S = t % 3 and spd set P = t % 2; units u = (key
    // block, query block) in the order (0,0), (0,1), (1,0), (1,1). The score
    // product of unit u + 1 is issued before the softmax of unit u, so the
    // matrix cores work while the vector ALUs do the softmax. Before the
    // softmax of the last unit the wave has issued every LDS read of stage S:
    // it waits for tile t + 1 (copied two steps ago, spd fetched one step
    // ago), meets the other waves at the barrier, refills stage S with tile
    // t + 3 and issues the first score product of tile t + 1.
    auto step = [&](int64_t t, auto stagec, auto setc) {
      constexpr int S = decltype(stagec)::value;
      constexpr int SN = (S + 1) % 3;
      constexpr int P = decltype(setc)::value;
      GT_FWD_STAGE(S, k_s, v_s)
      GT_FWD_STAGE(SN, k_n, v_n)
      auto& w = P == 0 ? wA : wB;
      auto& w_n = P == 0 ? wB : wA;
      if (!active) {
        // same loads, waits and barrier as the working waves
        spd_of(t + 2, w);
        wait_vmcnt<SPD_LOADS + Dma::NLOADS>();
        __builtin_amdgcn_s_barrier();
        copy_tile(t + 3, stagec);
        return;
      }
      bf16x8 vop[2][NCB];
      f32x16 s1, s2, s3;
      issue_scores<D, NKS>(sTab, w[1][0], lane4, k_s, off.k, 0, qf[1], s1);
      read_v<D>(v_s, off, 0, vop);
      softmax_pv<D, false>(s0, vop, kBC, sl2, sm[0], acc[0]);
      issue_scores<D, NKS>(sTab, w[0][1], lane4, k_s, off.k, 1, qf[0], s2);
      softmax_pv<D, false>(s1, vop, kBC, sl2, sm[1], acc[1]);
      issue_scores<D, NKS>(sTab, w[1][1], lane4, k_s, off.k, 1, qf[1], s3);
      read_v<D>(v_s, off, 1, vop);
      spd_of(t + 2, w);      // set P is free: tile t + 2's words
      sched_fence();
      softmax_pv<D, false>(s2, vop, kBC, sl2, sm[0], acc[0]);
      // Tile boundary: tile t + 1 must have landed; only tile t + 2's copy
      // (issued one step ago) and spd words (just issued) may be in flight.
      wait_vmcnt<SPD_LOADS + Dma::NLOADS>();
      __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0): this wave's LDS reads of stage S done
      __builtin_amdgcn_s_barrier();
      copy_tile(t + 3, stagec);
      sched_fence();
      issue_scores<D, NKS>(sTab, w_n[0][0], lane4, k_n, off.k, 0, qf[0], s0);
      softmax_pv<D, false>(s3, vop, kBC, sl2, sm[1], acc[1]);
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
    // one tile computed per step, every wait drains the loads.
    uint32_t w0[kQB][kKB][4], w1[kQB][kKB][4], w2[kQB][kKB][4];
    if (ntiles > 0) {
      copy_tile(0, S0());
      spd_of(0, w0);
      copy_tile(1, S1());
      spd_of(1, w1);
    }
    wait_vmcnt<0>();
    __syncthreads();     // table, and the copy of tile 0
    auto step = [&](int64_t t, auto stagec, auto maskc) {
      constexpr int S = decltype(stagec)::value;
      constexpr bool MASK = decltype(maskc)::value;
      GT_FWD_STAGE(S, k_s, v_s)
      copy_tile(t + 2, std::integral_constant<int, (S + 2) % 3>());
      spd_of(t + 2, S == 0 ? w2 : (S == 1 ? w0 : w1));
      sched_fence();
      auto& w = S == 0 ? w0 : (S == 1 ? w1 : w2);
      if (active) fwd_tile<D, NKS, MASK>(k_s, v_s, sTab, off, qf, w, lane4, a.Sk - t * kBC, sl2, sm, acc);
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
#undef GT_FWD_STAGE

  // Epilogue: O = O_acc / l, LSE = (m + log2 l) ln 2.
#pragma unroll
  for (int qb = 0; qb < kQB; ++qb) {
    const float lt = sm[qb].l + __shfl_xor(sm[qb].l, 32);
    const int64_t i = qbase + qb * 32 + col;
    if (i >= a.Sq || !item_ok) continue;
    float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
    float lse_out = lt > 0.0f ? (sm[qb].m + __log2f(lt)) * kLn2 : -INFINITY;
    float wo = 0.0f;     // weight of the running state (accumulate mode)
    if constexpr (OUT_F32) {
      if (a.accumulate) {
        float wb;
        lse_merge_weights(a.lse[(int64_t)h * a.Sq + i], lse_out, wo, wb, lse_out);
        inv *= wb;
      }
    }
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = cb * 32 + 8 * u + 4 * g;
        if (c >= DS) continue;                 // zero padding of a narrow head dim
        float o0 = acc[qb][cb][4 * u + 0] * inv, o1 = acc[qb][cb][4 * u + 1] * inv;
        float o2 = acc[qb][cb][4 * u + 2] * inv, o3 = acc[qb][cb][4 * u + 3] * inv;
        if constexpr (OUT_F32) {
          float* op = reinterpret_cast<float*>(a.o) + ((int64_t)h * a.Sq + i) * DS + c;
          if (wo != 0.0f) {
            const float4 old = *reinterpret_cast<const float4*>(op);
            o0 = fmaf(old.x, wo, o0);
            o1 = fmaf(old.y, wo, o1);
            o2 = fmaf(old.z, wo, o2);
            o3 = fmaf(old.w, wo, o3);
          }
          *reinterpret_cast<float4*>(op) = make_float4(o0, o1, o2, o3);
        } else {
          uint16_t* op = reinterpret_cast<uint16_t*>(a.o) + ((int64_t)h * a.Sq + i) * DS + c;
          uint2 pk;
          pk.x = (uint32_t)f2bf(o0) | ((uint32_t)f2bf(o1) << 16);
          pk.y = (uint32_t)f2bf(o2) | ((uint32_t)f2bf(o3) << 16);
          *reinterpret_cast<uint2*>(op) = pk;
        }
      }
    }
    if (g == 0) a.lse[(int64_t)h * a.Sq + i] = lse_out;
  }
}

// Vector-ALU path (fp32 inputs, any head dim): kValuSplit adjacent threads
// per query row, keys staged through LDS 128 at a time and split between
// them (thread s takes the KB-key block s of every tile), each with its own
// online softmax; the states are combined by lane shuffles at the end.
// fp32 math with the hardware exp2 and logf; o is fp32.
constexpr int kValuSplit = 16;
template <int D>
__global__ __launch_bounds__(128) void fwd_valu_kernel(FwdArgs a) {
  constexpr int KB = 128 / kValuSplit; // keys per thread per LDS tile
  constexpr int TK = KB * kValuSplit;
  constexpr int RPB = 128 / kValuSplit;
  constexpr int LR = valu_tile_rows<TK, KB>(), DP = valu_row_stride<D>();
  __shared__ __attribute__((aligned(16))) float sK[LR][DP];
  __shared__ __attribute__((aligned(16))) float sV[LR][DP];
  __shared__ float sT[256];
  const int tid = threadIdx.x;
  const int sp = tid % kValuSplit;   // this thread's key block of each tile
  const int64_t nqb = (a.Sq + RPB - 1) / RPB;
  const int h = (int)(blockIdx.x / nqb);
  const int64_t i = (blockIdx.x % nqb) * RPB + tid / kValuSplit;
  for (int t = tid; t < 256; t += 128)
    sT[t] = (t < a.n_buckets) ? a.table[(int64_t)table_row(a, h) * a.n_buckets + t] : 0.0f;
  const float* qg = reinterpret_cast<const float*>(a.q);
  const float* kg = reinterpret_cast<const float*>(a.k);
  const float* vg = reinterpret_cast<const float*>(a.v);
  const int64_t hq = (int64_t)h * a.Sq * D, hk = (int64_t)h * a.Sk * D;
  const bool ok = i < a.Sq;
  float qv[D], acc[D];
  load_row_f32<D>(qg + hq, ok ? i : 0, ok, a.scale, qv);
#pragma unroll
  for (int c = 0; c < D; ++c) acc[c] = 0.0f;
  const uint8_t* srow = ok ? seq_spd(a, h) + (a.row_off + i) * a.ld_spd + a.col_off : nullptr;
  float m = -INFINITY, l = 0.0f;     // running max (natural units) and sum relative to it
  // head dims up to 32: the next K/V tile is loaded into registers while
  // this one is computed (the barriers order LDS only)
  constexpr bool PF = D <= 32;
  RowPrefetchF32<TK, D, KB, 128> pf;
  if constexpr (PF) pf.load(kg + hk, vg + hk, 0, a.Sk);
  for (int64_t j0 = 0; j0 < a.Sk; j0 += TK) {
    lds_barrier();
    if constexpr (PF) {
      pf.store(sK, sV);
      if (j0 + TK < a.Sk) pf.load(kg + hk, vg + hk, j0 + TK, a.Sk);
    } else {
      stage_rows_f32<TK, D, KB, 128>(kg + hk, vg + hk, j0, a.Sk, sK, sV);
    }
    lds_barrier();
    const int nk = (int)((a.Sk - j0) < TK ? (a.Sk - j0) : TK);
    const int r0 = sp * KB;
    if (!ok || r0 >= nk) continue;
    // this thread's block of KB keys: their spd bytes in one load, one
    // running-max update
    uint32_t w[4];
    load_spd_block<KB>(srow, j0 + r0, a.Sk, a.spd_vec && r0 + KB <= nk, w);
    float sc[KB];
    float bm = -INFINITY;
#pragma unroll
    for (int r = 0; r < KB; ++r) {
      float x = sT[(w[r >> 2] >> (8 * (r & 3))) & 0xffu];
#pragma unroll
      for (int c = 0; c < D; ++c) x = fmaf(qv[c], sK[valu_row<KB>(r0 + r)][c], x);
      sc[r] = (r0 + r < nk) ? x : -INFINITY;
      bm = fmaxf(bm, sc[r]);
    }
    if (bm == -INFINITY) continue;
    if (bm > m) {
      const float alpha = (m == -INFINITY) ? 0.0f : exp2_fast((m - bm) * kLog2e);
      l *= alpha;
#pragma unroll
      for (int c = 0; c < D; ++c) acc[c] *= alpha;
      m = bm;
    }
#pragma unroll
    for (int r = 0; r < KB; ++r) {
      const float p = exp2_fast((sc[r] - m) * kLog2e);
      l += p;
#pragma unroll
      for (int c = 0; c < D; ++c) acc[c] = fmaf(p, sV[valu_row<KB>(r0 + r)][c], acc[c]);
    }
  }
  // combine the states of the row (adjacent lanes): max, then each
  // state scaled to it and summed
  float mall = m;
#pragma unroll
  for (int o = 1; o < kValuSplit; o <<= 1) mall = fmaxf(mall, __shfl_xor(mall, o));
  const float wgt = (m == -INFINITY) ? 0.0f : exp2_fast((m - mall) * kLog2e);
  l *= wgt;
#pragma unroll
  for (int o = 1; o < kValuSplit; o <<= 1) l += __shfl_xor(l, o);
#pragma unroll
  for (int c = 0; c < D; ++c) {
    acc[c] *= wgt;
#pragma unroll
    for (int o = 1; o < kValuSplit; o <<= 1) acc[c] += __shfl_xor(acc[c], o);
  }
  if (!ok) return;
  float inv = l > 0.0f ? 1.0f / l : 0.0f;
  float lse_out = l > 0.0f ? mall + logf(l) : -INFINITY;
  float wo = 0.0f;     // weight of the running state (accumulate mode)
  if (a.accumulate) {
    float wb;
    lse_merge_weights(a.lse[(int64_t)h * a.Sq + i], lse_out, wo, wb, lse_out);
    inv *= wb;
  }
  // every thread of the row writes the features c = sp mod kValuSplit; the first the LSE
  float* op = reinterpret_cast<float*>(a.o) + hq + i * D;
#pragma unroll
  for (int c = 0; c < D; ++c)
    if (c % kValuSplit == sp) op[c] = wo != 0.0f ? fmaf(op[c], wo, acc[c] * inv) : acc[c] * inv;
  if (sp == 0) a.lse[(int64_t)h * a.Sq + i] = lse_out;
}

template <int D, int DS, bool OUT_F32>
hipError_t launch_fwd_bf16(const FwdArgs& a, hipStream_t s) {
  constexpr int BR = kWaves * 32 * kQB;
  const int64_t nqb = (a.Sq + BR - 1) / BR;
  const dim3 grid((unsigned)(nqb * a.H));
  const bool skip = a.Sq % BR != 0;
  const int nseq = a.H / a.hpb;
  if constexpr (D == 32) {
    // batches of short sequences: two sequences per workgroup
    constexpr int BRP = kWaves / 2 * 32 * kQB;
    if (a.spd_vec && a.Sk % kBC == 0 && a.Sq <= BRP && a.hpb < a.H && nseq >= 2 && !a.accumulate) {
      const dim3 gridp((unsigned)((nseq + 1) / 2 * a.hpb));
      if (a.Sq % BRP != 0)
        hipLaunchKernelGGL((fwd_bf16_kernel<D, DS, OUT_F32, true, true, true, true>), gridp, dim3(kThreads), 0, s, a);
      else
        hipLaunchKernelGGL((fwd_bf16_kernel<D, DS, OUT_F32, true, true, false, true>), gridp, dim3(kThreads), 0, s, a);
      return hipGetLastError();
    }
  }
  if (a.spd_vec && a.Sk % kBC == 0) {
    if (skip)
      hipLaunchKernelGGL((fwd_bf16_kernel<D, DS, OUT_F32, true, true, true>), grid, dim3(kThreads), 0, s, a);
    else
      hipLaunchKernelGGL((fwd_bf16_kernel<D, DS, OUT_F32, true, true, false>), grid, dim3(kThreads), 0, s, a);
  } else if (a.spd_vec) {
    if (skip)
      hipLaunchKernelGGL((fwd_bf16_kernel<D, DS, OUT_F32, true, false, true>), grid, dim3(kThreads), 0, s, a);
    else
      hipLaunchKernelGGL((fwd_bf16_kernel<D, DS, OUT_F32, true, false, false>), grid, dim3(kThreads), 0, s, a);
  } else {
    if (skip)
      hipLaunchKernelGGL((fwd_bf16_kernel<D, DS, OUT_F32, false, false, true>), grid, dim3(kThreads), 0, s, a);
    else
      hipLaunchKernelGGL((fwd_bf16_kernel<D, DS, OUT_F32, false, false, false>), grid, dim3(kThreads), 0, s, a);
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_fwd(const FwdArgs& a, int d, bool bf16, bool out_f32, hipStream_t s) {
  // bf16 runs on the matrix cores at every head dim: 8 and 16 on 32-wide
  // tiles whose extra features are zero. fp32 runs on the vector ALUs.
  if (bf16) {
    if (!out_f32 && fwd_short_applies(a, d)) return launch_fwd_short_bf16(a, d, s);
    switch (d) {
      case 8: return out_f32 ? launch_fwd_bf16<32, 8, true>(a, s) : launch_fwd_bf16<32, 8, false>(a, s);
      case 16: return out_f32 ? launch_fwd_bf16<32, 16, true>(a, s) : launch_fwd_bf16<32, 16, false>(a, s);
      case 32: return out_f32 ? launch_fwd_bf16<32, 32, true>(a, s) : launch_fwd_bf16<32, 32, false>(a, s);
      default: return out_f32 ? launch_fwd_bf16<64, 64, true>(a, s) : launch_fwd_bf16<64, 64, false>(a, s);
    }
  }
  const dim3 grid((unsigned)((a.Sq + 128 / kValuSplit - 1) / (128 / kValuSplit) * a.H));
  switch (d) {
    case 8: hipLaunchKernelGGL((fwd_valu_kernel<8>), grid, dim3(128), 0, s, a); break;
    case 16: hipLaunchKernelGGL((fwd_valu_kernel<16>), grid, dim3(128), 0, s, a); break;
    case 32: hipLaunchKernelGGL((fwd_valu_kernel<32>), grid, dim3(128), 0, s, a); break;
    default: hipLaunchKernelGGL((fwd_valu_kernel<64>), grid, dim3(128), 0, s, a); break;
  }
  return hipGetLastError();
}

}  // namespace gt
