// Persistent forward for short sequences (bf16, head dims up to 32): see the
// kernel's description below. The building blocks are those of the full
// forward (fwd_tile.hpp).
#include "common.hpp"
#include "kernels.hpp"
#include "stage.hpp"
#include "fwd_tile.hpp"

namespace gt {

namespace {

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;

// Persistent forward for sequences of 33 to 256 rows with at most 127
// buckets (bf16 in and out, head dims 8, 16, 32 on 32-wide tiles; spd rows
// 4-byte aligned). Each wave owns 32 queries, so a workgroup covers a whole
// sequence, and the sequence's K and V (all rows) sit in LDS: one pair of
// barriers per sequence instead of one barrier per key tile. The per-lane
// bias table holds the byte values 0..127 (bytes of 128 or more are mapped
// to the padding entry 127, bias 0) and an entry of -inf (128) that masks
// the keys past N: with K and V that is 65 KB, so two workgroups share a
// compute unit and every SIMD runs four waves. The workgroups are
// persistent: workgroup w takes head (w mod hpb) of every (G / hpb)-th
// sequence, fills the table once, and loads the next sequence's K, V and Q
// rows into registers while it computes the current one. spd words stream
// two key blocks ahead across sequences (read 16 bytes at a time from 4-byte
// aligned offsets, through a resource that ends with the sequence's matrix);
// the score product of key block kb + 1 is issued before the softmax of
// block kb. TAIL: N is not a multiple of 32.
constexpr int kShortTabEntries = 129;
template <int DS, bool TAIL>
__global__ __launch_bounds__(kThreads, 2) void fwd_short_bf16_kernel(FwdArgs a) {
  constexpr int D = 32;
  constexpr int NKC = D / 16;
  constexpr int NKS = (DS + 15) / 16;
  constexpr int NCB = D / 32;
  constexpr int ROWS = 256;
  constexpr int CPS = DS / 8;                   // 16-byte chunks per source row
  constexpr int PER = ROWS * CPS;               // chunks per tensor (a multiple of 64)
  constexpr int IPT = (PER + kThreads - 1) / kThreads;
  __shared__ __attribute__((aligned(16))) uint16_t sK[ROWS * D], sV[ROWS * D];
  __shared__ __attribute__((aligned(16))) float sTab[kShortTabEntries * 64];

  const int tid = threadIdx.x;
  const int lane = tid & 63, w = wave_id();
  const int col = lane & 31, g = lane >> 5;
  const uint32_t lane4 = (uint32_t)lane * 4u;
  const int N = (int)a.Sq;
  const int nkb = (N + 31) / 32;                // at least 2
  const int G = (int)gridDim.x;
  const int lw = (int)xcd_remap(blockIdx.x, G);
  const int head = lw % a.hpb;
  const int slot = lw / a.hpb;
  const int nslots = G / a.hpb;
  const int nseq = a.H / a.hpb;
  const float sl2 = a.scale * kLog2e;
  const int ld = (int)a.ld_spd;
  const int qi = w * 32 + col;                  // this lane's query
  const int qc = qi < N ? qi : N - 1;
  const bool wact = w * 32 < N;
  const FwdOffsets<D> off;

  // table entry (b, lane) at float 64 b + lane: bias / scale for b below
  // n_buckets, 0 up to 127, -inf at 128; zero K, V (features past the head
  // dim stay zero)
  {
    const float inv_scale = 1.0f / a.scale;
    const float* th = a.table + (int64_t)head * a.n_buckets;
    for (int t = tid; t < kShortTabEntries * 16; t += kThreads) {
      const int bk = t >> 4;
      const float x = bk < 128 ? (bk < a.n_buckets ? th[bk] * inv_scale : 0.0f) : -INFINITY;
      reinterpret_cast<float4*>(sTab)[t] = make_float4(x, x, x, x);
    }
    for (int t = tid; t < ROWS * D / 8; t += kThreads) {
      reinterpret_cast<uint4*>(sK)[t] = make_uint4(0u, 0u, 0u, 0u);
      reinterpret_cast<uint4*>(sV)[t] = make_uint4(0u, 0u, 0u, 0u);
    }
  }

  // Loads of sequence s into registers: its K and V rows (item u = row *
  // DS/8 + chunk, thread u mod 512; rows past N read zero) and this lane's
  // Q row.
  uint4 rk[IPT], rv[IPT];
  bf16x8 qf[NKC], qn[NKC];
  auto issue = [&](int s) {
    const int h = s * a.hpb + head;
    const int64_t rowbase = (int64_t)h * N * DS;
    const int64_t nbytes = (int64_t)N * DS * 2;
    const __amdgpu_buffer_rsrc_t sk = make_rsrc_n(reinterpret_cast<const uint16_t*>(a.k) + rowbase, nbytes);
    const __amdgpu_buffer_rsrc_t sv = make_rsrc_n(reinterpret_cast<const uint16_t*>(a.v) + rowbase, nbytes);
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int u = tid + i * kThreads;
      if (u < PER) {
        const uint32_t vo = (uint32_t)((u / CPS) * DS * 2 + (u % CPS) * 16);
        rk[i] = buf_b128(sk, vo);
        rv[i] = buf_b128(sv, vo);
      }
    }
    const uint16_t* qh = reinterpret_cast<const uint16_t*>(a.q) + rowbase;
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc)
      qn[kc] = (kc * 16 + g * 8 < DS) ? *reinterpret_cast<const bf16x8*>(qh + (int64_t)qc * DS + kc * 16 + g * 8)
                                      : zero_bf16x8();
  };
  auto spd_rs = [&](int s) {
    const int h = s * a.hpb + head;
    return make_rsrc_n(seq_spd(a, h), (int64_t)N * ld);
  };
  const uint32_t voff = (uint32_t)(qc * ld + 16 * g);
  // Bucket words of key block kb as table entries: bytes of 128 or more to
  // the padding entry 127; with TAIL, keys past N to the -inf entry.
  auto entries = [&](const uint32_t (&wsrc)[4], int kb, uint32_t (&e)[4]) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      e[u] = wsrc[u];
      opaque(e[u]);
    }
    if (__any(((e[0] | e[1] | e[2] | e[3]) & 0x80808080u) != 0)) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        uint32_t x = e[u];
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if ((x >> (8 * k + 7)) & 1u) x = (x & ~(0xffu << (8 * k))) | (0x7fu << (8 * k));
        e[u] = x;
      }
    }
    if constexpr (TAIL) {
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (kb * 32 + 16 * g + 4 * u >= N) e[u] = 0x80808080u;   // N is a multiple of 4
    }
  };

  SoftmaxState st;
  f32x16 acc[NCB];
  uint32_t wd[3][4];                              // spd words of key blocks kb, kb + 1, kb + 2

  // One sequence: its K, V, Q are in registers on entry (loaded during the
  // previous one), and wd[0], wd[1] hold its first spd words. The spd words
  // stream over (sequence, key block) two blocks ahead: past the last block
  // come blocks 0 and 1 of the next sequence.
  auto run = [&](int s) {
    const int nxt = s + nslots < nseq ? s + nslots : s;
    const __amdgpu_buffer_rsrc_t rs = spd_rs(s);
    const __amdgpu_buffer_rsrc_t rn = spd_rs(nxt);
    __syncthreads();            // the previous sequence's reads of K and V are done
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int u = tid + i * kThreads;
      if (u < PER) {
        const int row = u / CPS, chunk = u % CPS;
        const int lo = row * D + swz_tile<D>(row, chunk) * 8;
        *reinterpret_cast<uint4*>(sK + lo) = rk[i];
        *reinterpret_cast<uint4*>(sV + lo) = rv[i];
      }
    }
#pragma unroll
    for (int kc = 0; kc < NKC; ++kc) qf[kc] = qn[kc];
    __syncthreads();            // K, V of this sequence visible
    issue(nxt);
    sched_fence();
    st.m = -INFINITY;
    st.mneg = 0.0f;
    st.l = 0.0f;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[cb] = zero_f32x16();
    f32x16 sc;
    if (wact) {
      uint32_t e[4];
      entries(wd[0], 0, e);
      issue_scores<D, NKS>(sTab, e, lane4, sK, off.k, 0, qf, sc);
    }
#pragma unroll
    for (int kb = 0; kb < ROWS / 32; ++kb) {
      if (kb < nkb) {
        // words of block kb + 2 (of the next sequence past the end)
        {
          const int kf = kb + 2;
          uint32_t* dst = wd[(kb + 2) % 3];
          if (kf < nkb)
            buf_u128(rs, voff, (uint32_t)(kf * 32), dst);
          else
            buf_u128(rn, voff, (uint32_t)((kf - nkb) * 32), dst);
        }
        sched_fence();
        if (wact) {
          // next block's scores, also past the last block (its K rows are the
          // zero rows of the last copied tile or unused LDS, and the result
          // is never read), so that the accumulator is never copied
          f32x16 sn;
          {
            uint32_t e[4];
            entries(wd[(kb + 1) % 3], kb + 1, e);
            issue_scores<D, NKS>(sTab, e, lane4, sK, off.k, (kb + 1) & 7, qf, sn);
          }
          bf16x8 vop[2][NCB];
          read_v<D>(sV, off, kb, vop);
          softmax_pv<D, false>(sc, vop, 32, sl2, st, acc);
          sc = sn;
        }
      }
    }
    // the next sequence's first two word sets sit in wd[nkb % 3], wd[(nkb + 1) % 3]
    if (nkb % 3 == 1) {
#pragma unroll
      for (int e = 0; e < 4; ++e) { const uint32_t t0 = wd[0][e]; wd[0][e] = wd[1][e]; wd[1][e] = wd[2][e]; wd[2][e] = t0; }
    } else if (nkb % 3 == 2) {
#pragma unroll
      for (int e = 0; e < 4; ++e) { const uint32_t t2 = wd[2][e]; wd[2][e] = wd[1][e]; wd[1][e] = wd[0][e]; wd[0][e] = t2; }
    }
    // epilogue: O = O_acc / l, LSE = (m + log2 l) ln 2
    if (wact) {
      const float lt = st.l + __shfl_xor(st.l, 32);
      if (qi < N) {
        const int h = s * a.hpb + head;
        const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
        const float lse_out = lt > 0.0f ? (st.m + __log2f(lt)) * kLn2 : -INFINITY;
        uint16_t* op = reinterpret_cast<uint16_t*>(a.o) + ((int64_t)h * N + qi) * DS;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int c = 8 * u + 4 * g;
          if (c >= DS) continue;
          uint2 pk;
          pk.x = (uint32_t)f2bf(acc[0][4 * u] * inv) | ((uint32_t)f2bf(acc[0][4 * u + 1] * inv) << 16);
          pk.y = (uint32_t)f2bf(acc[0][4 * u + 2] * inv) | ((uint32_t)f2bf(acc[0][4 * u + 3] * inv) << 16);
          *reinterpret_cast<uint2*>(op + c) = pk;
        }
        if (g == 0) a.lse[(int64_t)h * N + qi] = lse_out;
      }
    }
  };

  issue(slot);
  {
    const __amdgpu_buffer_rsrc_t rs = spd_rs(slot);
    buf_u128(rs, voff, 0u, wd[0]);
    buf_u128(rs, voff, 32u, wd[1]);
  }
  for (int s = slot; s < nseq; s += nslots) run(s);
  wait_vmcnt<0>();     // drain the loads issued for the last (repeated) sequence
}

template <int DS>
void launch_short_t(const FwdArgs& a, hipStream_t s) {
  const int nseq = a.H / a.hpb;
  // two workgroups per compute unit where the registers allow four waves per SIMD
  int slots = (DS <= 16 ? 512 : 256) / a.hpb;
  if (slots < 1) slots = 1;
  if (slots > nseq) slots = nseq;
  const dim3 grid((unsigned)(slots * a.hpb));
  if (a.Sq % 32 != 0)
    hipLaunchKernelGGL((fwd_short_bf16_kernel<DS, true>), grid, dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((fwd_short_bf16_kernel<DS, false>), grid, dim3(kThreads), 0, s, a);
}

}  // namespace

bool fwd_short_applies(const FwdArgs& a, int d) {
  return d <= 32 && !a.accumulate && a.row_off == 0 && a.col_off == 0 && a.Sq == a.Sk &&
         a.Sq > 32 && a.Sq <= 256 && a.n_buckets <= 127 && a.hpb >= 1 && a.H % a.hpb == 0 &&
         reinterpret_cast<uintptr_t>(a.spd) % 4 == 0 && a.ld_spd % 4 == 0 && a.spd_bstride % 4 == 0;
}

hipError_t launch_fwd_short_bf16(const FwdArgs& a, int d, hipStream_t s) {
  switch (d) {
    case 8: launch_short_t<8>(a, s); break;
    case 16: launch_short_t<16>(a, s); break;
    default: launch_short_t<32>(a, s); break;
  }
  return hipGetLastError();
}

}  // namespace gt
