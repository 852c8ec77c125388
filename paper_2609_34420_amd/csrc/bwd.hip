// Backward kernels of biased attention.
//
// With P = softmax(S), S = scale Q K^T + B (Eq. (1)) and L = sum(O * dO):
//   Dlt_i = sum_c dO_ic O_ic,  dS = P * (dO V^T - Dlt),
//   dV = P^T dO,  dK = scale dS^T Q,  dQ = scale dS K,
//   dtable[h, b] = sum of dS_ij over pairs with spd_ij = b.
// P is recomputed from the saved LSE, never stored.
//
// Launch order: prepare (lse2 = LSE log2 e, +inf for an empty row so that
// P = 0; Dlt; dtable = 0), then the key-stationary dK/dV/dtable kernel and
// the query-stationary dQ kernel (bwd_dkdv.hip, bwd_dq.hip for bf16 at
// every head dim; the vector-ALU kernels below for fp32). Splitting dQ from
// dK/dV recomputes two products but needs no atomics on dQ. Sequences of at
// most 256 rows at head dims up to 32 take one fused kernel instead, which
// also does the prepare stage's work (bwd_short.hip): there a workgroup holds
// every key, so dQ is reduced inside it.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace gt {

namespace {

// ---------------------------------------------------------------------------
// Preprocess: lse2, Dlt; dtable = 0.
// ---------------------------------------------------------------------------
// Preprocess, grid (ceil(max(Sq, Sk)/256), H): per query row lse2 = LSE log2 e
// (+inf for an empty row), Dlt = rowsum(dO * O); per block of 256 rows the
// largest squared norms of dO rows (query side) and V rows (key side) and the
// largest |Dlt|: the dK/dV stage bounds |dS| with them. Block (0, 0) also
// zeroes dtable unless the call accumulates.
template <int D, bool BF16>
__global__ __launch_bounds__(256) void bwd_prep_kernel(BwdArgs a) {
  // A row is read by TPR consecutive lanes, 16 bytes each, so a wave's loads
  // cover whole rows contiguously; the block's 256 rows take TPR passes.
  constexpr int EPC = BF16 ? 8 : 4;          // elements per 16-byte chunk
  constexpr int TPR = D / EPC;               // lanes per row
  constexpr int RPP = 256 / TPR;             // rows per pass
  __shared__ float red[3][4];
  const int h = blockIdx.y;
  const int sub = threadIdx.x % TPR;
  if (blockIdx.x == 0 && blockIdx.y == 0 && !a.accumulate) {
    for (int t = threadIdx.x; t < a.hpb * a.n_buckets; t += 256) a.dtable[t] = 0.0f;
  }
  // dot products of one 16-byte chunk
  auto chunk_dot = [](const void* x, const void* y, float& xy, float& yy) {
    if constexpr (BF16) {
      const uint4 xv = *reinterpret_cast<const uint4*>(x);
      const uint4 yv = *reinterpret_cast<const uint4*>(y);
      const uint16_t* xp = reinterpret_cast<const uint16_t*>(&xv);
      const uint16_t* yp = reinterpret_cast<const uint16_t*>(&yv);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float yf = bf2f(yp[e]);
        xy = fmaf(bf2f(xp[e]), yf, xy);
        yy = fmaf(yf, yf, yy);
      }
    } else {
      const float4 xv = *reinterpret_cast<const float4*>(x);
      const float4 yv = *reinterpret_cast<const float4*>(y);
      xy = fmaf(xv.x, yv.x, fmaf(xv.y, yv.y, fmaf(xv.z, yv.z, fmaf(xv.w, yv.w, xy))));
      yy = fmaf(yv.x, yv.x, fmaf(yv.y, yv.y, fmaf(yv.z, yv.z, fmaf(yv.w, yv.w, yy))));
    }
  };
  using T = std::conditional_t<BF16, uint16_t, float>;
  float nd = 0.0f, nv = 0.0f, nl = 0.0f;
#pragma unroll
  for (int pass = 0; pass < TPR; ++pass) {
    const int64_t i = (int64_t)blockIdx.x * 256 + pass * RPP + threadIdx.x / TPR;
    float acc = 0.0f, sq = 0.0f, vq = 0.0f, unused = 0.0f;
    if (i < a.Sq) {
      const int64_t off = ((int64_t)h * a.Sq + i) * D + sub * EPC;
      chunk_dot(reinterpret_cast<const T*>(a.o) + off, reinterpret_cast<const T*>(a.d_o) + off, acc, sq);
    }
    if (i < a.Sk) {
      const int64_t off = ((int64_t)h * a.Sk + i) * D + sub * EPC;
      const T* v = reinterpret_cast<const T*>(a.v) + off;
      chunk_dot(v, v, unused, vq);
    }
#pragma unroll
    for (int o = TPR / 2; o >= 1; o >>= 1) {
      acc += __shfl_xor(acc, o);
      sq += __shfl_xor(sq, o);
      vq += __shfl_xor(vq, o);
    }
    if (i < a.Sq) {
      const int64_t row = (int64_t)h * a.Sq + i;
      nd = fmaxf(nd, sq);
      nl = fmaxf(nl, fabsf(acc));
      if (sub == 0) {
        a.dlt[row] = acc;
        const float L = a.lse[row];
        a.lse2[row] = (L == -INFINITY) ? INFINITY : L * kLog2e;
      }
    }
    if (i < a.Sk) nv = fmaxf(nv, vq);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    nd = fmaxf(nd, __shfl_xor(nd, off));
    nv = fmaxf(nv, __shfl_xor(nv, off));
    nl = fmaxf(nl, __shfl_xor(nl, off));
  }
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[0][wave] = nd;
    red[1][wave] = nv;
    red[2][wave] = nl;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const int64_t nblk = gridDim.x;
    float* out = a.nmax + ((int64_t)h * nblk + blockIdx.x) * 4;
    out[0] = fmaxf(fmaxf(red[0][0], red[0][1]), fmaxf(red[0][2], red[0][3]));
    out[1] = fmaxf(fmaxf(red[1][0], red[1][1]), fmaxf(red[1][2], red[1][3]));
    out[2] = fmaxf(fmaxf(red[2][0], red[2][1]), fmaxf(red[2][2], red[2][3]));
    out[3] = 0.0f;
  }
}

// Preprocess for sequences of at most 256 rows (one row block per head):
// one wave per head, so the head's maxima are reduced within the wave (no
// LDS, no barrier) and a workgroup of 4 waves covers 4 heads. The outputs
// are those of bwd_prep_kernel with one 256-row block.
template <int D, bool BF16>
__global__ __launch_bounds__(256) void bwd_prep_short_kernel(BwdArgs a) {
  constexpr int EPC = BF16 ? 8 : 4;
  constexpr int TPR = D / EPC;               // lanes per row
  constexpr int RPW = 64 / TPR;              // rows per wave pass
  constexpr int NPASS = 256 / RPW;
  const int lane = threadIdx.x & 63;
  const int h = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (blockIdx.x == 0 && !a.accumulate) {
    for (int t = threadIdx.x; t < a.hpb * a.n_buckets; t += 256) a.dtable[t] = 0.0f;
  }
  if (h >= a.H) return;
  const int sub = lane % TPR;
  using T = std::conditional_t<BF16, uint16_t, float>;
  auto chunk_dot = [](const T* x, const T* y, float& xy, float& yy) {
    if constexpr (BF16) {
      const uint4 xv = *reinterpret_cast<const uint4*>(x);
      const uint4 yv = *reinterpret_cast<const uint4*>(y);
      const uint16_t* xp = reinterpret_cast<const uint16_t*>(&xv);
      const uint16_t* yp = reinterpret_cast<const uint16_t*>(&yv);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float yf = bf2f(yp[e]);
        xy = fmaf(bf2f(xp[e]), yf, xy);
        yy = fmaf(yf, yf, yy);
      }
    } else {
      const float4 xv = *reinterpret_cast<const float4*>(x);
      const float4 yv = *reinterpret_cast<const float4*>(y);
      xy = fmaf(xv.x, yv.x, fmaf(xv.y, yv.y, fmaf(xv.z, yv.z, fmaf(xv.w, yv.w, xy))));
      yy = fmaf(yv.x, yv.x, fmaf(yv.y, yv.y, fmaf(yv.z, yv.z, fmaf(yv.w, yv.w, yy))));
    }
  };
  float nd = 0.0f, nv = 0.0f, nl = 0.0f;
#pragma unroll 4
  for (int pass = 0; pass < NPASS; ++pass) {
    const int64_t i = pass * RPW + lane / TPR;
    float acc = 0.0f, sq = 0.0f, vq = 0.0f, unused = 0.0f;
    if (i < a.Sq) {
      const int64_t off = ((int64_t)h * a.Sq + i) * D + sub * EPC;
      chunk_dot(reinterpret_cast<const T*>(a.o) + off, reinterpret_cast<const T*>(a.d_o) + off, acc, sq);
    }
    if (i < a.Sk) {
      const int64_t off = ((int64_t)h * a.Sk + i) * D + sub * EPC;
      const T* v = reinterpret_cast<const T*>(a.v) + off;
      chunk_dot(v, v, unused, vq);
    }
#pragma unroll
    for (int o = TPR / 2; o >= 1; o >>= 1) {
      acc += __shfl_xor(acc, o);
      sq += __shfl_xor(sq, o);
      vq += __shfl_xor(vq, o);
    }
    if (i < a.Sq) {
      const int64_t row = (int64_t)h * a.Sq + i;
      nd = fmaxf(nd, sq);
      nl = fmaxf(nl, fabsf(acc));
      if (sub == 0) {
        a.dlt[row] = acc;
        const float L = a.lse[row];
        a.lse2[row] = (L == -INFINITY) ? INFINITY : L * kLog2e;
      }
    }
    if (i < a.Sk) nv = fmaxf(nv, vq);
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    nd = fmaxf(nd, __shfl_xor(nd, off));
    nv = fmaxf(nv, __shfl_xor(nv, off));
    nl = fmaxf(nl, __shfl_xor(nl, off));
  }
  if (lane == 0) {
    float* out = a.nmax + (int64_t)h * 4;
    out[0] = nd;
    out[1] = nv;
    out[2] = nl;
    out[3] = 0.0f;
  }
}

// ---------------------------------------------------------------------------
// Vector-ALU path (fp32 inputs): one thread per query row / key column, fp32
// math; dq, dk, dv are fp32 (stored, or added into the caller's
// accumulators).
// ---------------------------------------------------------------------------
__device__ __forceinline__ void store_grad(float* base, int64_t idx, float x, bool accumulate) {
  if (accumulate)
    base[idx] += x;
  else
    base[idx] = x;
}

// The vector-ALU kernels split each row's loop between kValuSplit adjacent
// threads (keys for dQ, queries for dK / dV) and add their partial sums by
// lane shuffles at the end.
constexpr int kValuSplit = 16;

template <int D>
__global__ __launch_bounds__(128) void bwd_dq_valu_kernel(BwdArgs a) {
  constexpr int KB = 128 / kValuSplit; // keys per thread per LDS tile
  constexpr int TK = KB * kValuSplit;
  constexpr int RPB = 128 / kValuSplit;
  constexpr int LR = valu_tile_rows<TK, KB>(), DP = valu_row_stride<D>();
  __shared__ __attribute__((aligned(16))) float sK[LR][DP];
  __shared__ __attribute__((aligned(16))) float sV[LR][DP];
  __shared__ float sT[256];
  // dtable histogram in fp32: LDS float atomics are slow, but fp32 inputs
  // need the unquantised dS
  __shared__ float sH[256];
  const int tid = threadIdx.x;
  const int sp = tid % kValuSplit;   // this thread's key block of each tile
  const int64_t nqb = (a.Sq + RPB - 1) / RPB;
  const int h = (int)(blockIdx.x / nqb);
  const int64_t i = (blockIdx.x % nqb) * RPB + tid / kValuSplit;
  for (int t = tid; t < 256; t += 128) {
    sT[t] = (t < a.n_buckets) ? a.table[(int64_t)table_row(a, h) * a.n_buckets + t] : 0.0f;
    sH[t] = 0.0f;
  }
  const float* qg = reinterpret_cast<const float*>(a.q);
  const float* kg = reinterpret_cast<const float*>(a.k);
  const float* vg = reinterpret_cast<const float*>(a.v);
  const float* dog = reinterpret_cast<const float*>(a.d_o);
  const int64_t hq = (int64_t)h * a.Sq * D, hk = (int64_t)h * a.Sk * D;
  const bool ok = i < a.Sq;
  float qv[D], dov[D], acc[D];
  load_row_f32<D>(qg + hq, ok ? i : 0, ok, a.scale, qv);
  load_row_f32<D>(dog + hq, ok ? i : 0, ok, 1.0f, dov);
#pragma unroll
  for (int c = 0; c < D; ++c) acc[c] = 0.0f;
  const float L = ok ? a.lse[(int64_t)h * a.Sq + i] : -INFINITY;
  const float dlt = ok ? a.dlt[(int64_t)h * a.Sq + i] : 0.0f;
  const uint8_t* srow = ok ? seq_spd(a, h) + (a.row_off + i) * a.ld_spd + a.col_off : nullptr;
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
    if (!ok || L == -INFINITY || r0 >= nk) continue;
    // this thread's block of KB keys: their spd bytes in one load
    uint32_t w[4];
    load_spd_block<KB>(srow, j0 + r0, a.Sk, a.spd_vec && r0 + KB <= nk, w);
    const int nr = nk - r0 < KB ? nk - r0 : KB;
    for (int r = 0; r < nr; ++r) {
      const int key = r0 + r;
      const int lr = valu_row<KB>(key);
      float sc = 0.0f, dp = 0.0f;
#pragma unroll
      for (int c = 0; c < D; ++c) {
        sc = fmaf(qv[c], sK[lr][c], sc);
        dp = fmaf(dov[c], sV[lr][c], dp);
      }
      const uint32_t b = (w[r >> 2] >> (8 * (r & 3))) & 0xffu;
      const float p = exp2_fast((sc + sT[b] - L) * kLog2e);
      const float ds = p * (dp - dlt);
#pragma unroll
      for (int c = 0; c < D; ++c) acc[c] = fmaf(ds, sK[lr][c], acc[c]);
      if (b < (uint32_t)a.n_buckets) atomicAdd(&sH[b], ds);
    }
  }
  // the row's partial sums (adjacent lanes)
#pragma unroll
  for (int c = 0; c < D; ++c)
#pragma unroll
    for (int o = 1; o < kValuSplit; o <<= 1) acc[c] += __shfl_xor(acc[c], o);
  if (ok) {
#pragma unroll
    for (int c = 0; c < D; ++c)
      if (c % kValuSplit == sp)
        store_grad(reinterpret_cast<float*>(a.dq), hq + i * D + c, acc[c] * a.scale, a.accumulate);
  }
  __syncthreads();
  float* dth = a.dtable + (int64_t)table_row(a, h) * a.n_buckets;
  for (int t = tid; t < a.n_buckets; t += 128)
    if (sH[t] != 0.0f) atomicAdd(&dth[t], sH[t]);
}

template <int D>
__global__ __launch_bounds__(128) void bwd_dkdv_valu_kernel(BwdArgs a) {
  constexpr int QB = 64 / kValuSplit;  // queries per thread per LDS tile
  constexpr int TQ = QB * kValuSplit;
  constexpr int RPB = 128 / kValuSplit;
  constexpr int LR = valu_tile_rows<TQ, QB>(), DP = valu_row_stride<D>();
  __shared__ __attribute__((aligned(16))) float sQ[LR][DP];
  __shared__ __attribute__((aligned(16))) float sO[LR][DP];
  __shared__ float sL[TQ], sD[TQ];
  __shared__ float sT[256];
  __shared__ uint8_t sS[TQ][RPB];    // spd of the tile's queries x this workgroup's keys
  const int tid = threadIdx.x;
  const int sp = tid % kValuSplit;   // this thread's queries of each tile
  const int64_t nkb = (a.Sk + RPB - 1) / RPB;
  const int h = (int)(blockIdx.x / nkb);
  const int64_t jb = (blockIdx.x % nkb) * RPB;
  const int jl = tid / kValuSplit;   // this thread's key within the workgroup
  const int64_t j = jb + jl;
  for (int t = tid; t < 256; t += 128)
    sT[t] = (t < a.n_buckets) ? a.table[(int64_t)table_row(a, h) * a.n_buckets + t] : 0.0f;
  const int64_t hq = (int64_t)h * a.Sq * D, hk = (int64_t)h * a.Sk * D;
  const uint8_t* sbase = seq_spd(a, h) + a.row_off * a.ld_spd + a.col_off;
  const bool ok = j < a.Sk;
  float kv[D], vv[D], dk[D], dv[D];
  load_row_f32<D>(reinterpret_cast<const float*>(a.k) + hk, ok ? j : 0, ok, a.scale, kv);
  load_row_f32<D>(reinterpret_cast<const float*>(a.v) + hk, ok ? j : 0, ok, 1.0f, vv);
#pragma unroll
  for (int c = 0; c < D; ++c) {
    dk[c] = 0.0f;
    dv[c] = 0.0f;
  }
  // A tile: Q and dO rows, LSE and Dlt, and the spd bytes of its queries x
  // this workgroup's keys (issued together rather than one per score). At
  // head dims up to 32 the next tile is loaded into registers while this one
  // is computed (the barriers order LDS only).
  const float* qf = reinterpret_cast<const float*>(a.q) + hq;
  const float* of = reinterpret_cast<const float*>(a.d_o) + hq;
  constexpr bool PF = D <= 32;
  constexpr int NSB = TQ * RPB / 128;          // spd bytes per thread per tile
  static_assert(TQ <= 128 && (TQ * RPB) % 128 == 0, "tile statistics and spd bytes per thread");
  RowPrefetchF32<TQ, D, QB, 128> pf;
  float pl = -INFINITY, pd = 0.0f;
  uint8_t psb[NSB];
  auto load_small = [&](int64_t i0) {
    const bool in = tid < TQ && i0 + tid < a.Sq;
    pl = in ? a.lse[(int64_t)h * a.Sq + i0 + tid] : -INFINITY;
    pd = in ? a.dlt[(int64_t)h * a.Sq + i0 + tid] : 0.0f;
#pragma unroll
    for (int s = 0; s < NSB; ++s) {
      const int t = tid + 128 * s, r = t / RPB, c = t % RPB;
      psb[s] = (i0 + r < a.Sq && jb + c < a.Sk) ? sbase[(i0 + r) * a.ld_spd + jb + c] : (uint8_t)0;
    }
  };
  auto store_small = [&]() {
    if (tid < TQ) {
      sL[tid] = pl;
      sD[tid] = pd;
    }
#pragma unroll
    for (int s = 0; s < NSB; ++s) {
      const int t = tid + 128 * s;
      sS[t / RPB][t % RPB] = psb[s];
    }
  };
  if constexpr (PF) {
    pf.load(qf, of, 0, a.Sq);
    load_small(0);
  }
  for (int64_t i0 = 0; i0 < a.Sq; i0 += TQ) {
    lds_barrier();
    if constexpr (PF) {
      pf.store(sQ, sO);
      store_small();
      if (i0 + TQ < a.Sq) {
        pf.load(qf, of, i0 + TQ, a.Sq);
        load_small(i0 + TQ);
      }
    } else {
      stage_rows_f32<TQ, D, QB, 128>(qf, of, i0, a.Sq, sQ, sO);
      load_small(i0);
      store_small();
    }
    lds_barrier();
    if (!ok) continue;
    const int nq = (int)((a.Sq - i0) < TQ ? (a.Sq - i0) : TQ);
    const int e = (sp + 1) * QB < nq ? (sp + 1) * QB : nq;
    for (int r = sp * QB; r < e; ++r) {
      if (sL[r] == -INFINITY) continue;
      const int lr = valu_row<QB>(r);
      float s = 0.0f, dp = 0.0f;
#pragma unroll
      for (int c = 0; c < D; ++c) {
        s = fmaf(sQ[lr][c], kv[c], s);
        dp = fmaf(sO[lr][c], vv[c], dp);
      }
      const float p = exp2_fast((s + sT[sS[r][jl]] - sL[r]) * kLog2e);
      const float ds = p * (dp - sD[r]);
#pragma unroll
      for (int c = 0; c < D; ++c) {
        dv[c] = fmaf(p, sO[lr][c], dv[c]);
        dk[c] = fmaf(ds, sQ[lr][c], dk[c]);
      }
    }
  }
  // the key's partial sums (adjacent lanes)
#pragma unroll
  for (int c = 0; c < D; ++c)
#pragma unroll
    for (int o = 1; o < kValuSplit; o <<= 1) {
      dk[c] += __shfl_xor(dk[c], o);
      dv[c] += __shfl_xor(dv[c], o);
    }
  if (!ok) return;
#pragma unroll
  for (int c = 0; c < D; ++c) {
    if (c % kValuSplit != sp) continue;
    store_grad(reinterpret_cast<float*>(a.dk), hk + j * D + c, dk[c] * a.scale, a.accumulate);
    store_grad(reinterpret_cast<float*>(a.dv), hk + j * D + c, dv[c], a.accumulate);
  }
}

template <int D>
hipError_t launch_bwd_t(const BwdArgs& a, bool bf16, int phase, hipStream_t s) {
  hipError_t e = hipSuccess;
  // sequences of at most 256 rows: one fused kernel, prepare stage included
  if (bf16 && phase < 0 && bwd_short_applies(a, D)) return launch_bwd_short_bf16(a, D, s);
  if (phase < 0 || phase == 0) {
    const int64_t rows = a.Sq > a.Sk ? a.Sq : a.Sk;
    if (rows <= 256) {
      const dim3 grid((unsigned)((a.H + 3) / 4));
      if (bf16)
        hipLaunchKernelGGL((bwd_prep_short_kernel<D, true>), grid, dim3(256), 0, s, a);
      else
        hipLaunchKernelGGL((bwd_prep_short_kernel<D, false>), grid, dim3(256), 0, s, a);
    } else {
      const dim3 grid((unsigned)((rows + 255) / 256), (unsigned)a.H);
      if (bf16)
        hipLaunchKernelGGL((bwd_prep_kernel<D, true>), grid, dim3(256), 0, s, a);
      else
        hipLaunchKernelGGL((bwd_prep_kernel<D, false>), grid, dim3(256), 0, s, a);
    }
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (bf16) {     // matrix cores at every head dim (8 and 16 on 32-wide tiles)
    if (phase < 0 || phase == 1) {
      if ((e = launch_dkdv_bf16(a, D, s)) != hipSuccess) return e;
    }
    if (phase < 0 || phase == 2) {
      if ((e = launch_dq_bf16(a, D, s)) != hipSuccess) return e;
    }
    return e;
  }
  // vector-ALU path (fp32): dK/dV in phase 1, dQ and dtable in phase 2
  constexpr int RPB = 128 / kValuSplit;
  const int64_t nkb = (a.Sk + RPB - 1) / RPB, nqb = (a.Sq + RPB - 1) / RPB;
  if (phase < 0 || phase == 1) {
    hipLaunchKernelGGL((bwd_dkdv_valu_kernel<D>), dim3((unsigned)(nkb * a.H)), dim3(128), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (phase < 0 || phase == 2) {
    hipLaunchKernelGGL((bwd_dq_valu_kernel<D>), dim3((unsigned)(nqb * a.H)), dim3(128), 0, s, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return e;
}

}  // namespace

hipError_t launch_bwd(const BwdArgs& a, int d, bool bf16, int phase, hipStream_t s) {
  switch (d) {
    case 8: return launch_bwd_t<8>(a, bf16, phase, s);
    case 16: return launch_bwd_t<16>(a, bf16, phase, s);
    case 32: return launch_bwd_t<32>(a, bf16, phase, s);
    default: return launch_bwd_t<64>(a, bf16, phase, s);
  }
}

}  // namespace gt
