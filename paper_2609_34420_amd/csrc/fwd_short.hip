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
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// x as three bf16 terms hi + mid + lo (exact to about 2^-24 of |x|; -inf
// gives hi = -inf and zero terms).
__device__ __forceinline__ void split3(float x, __bf16& h, __bf16& m, __bf16& l) {
  h = (__bf16)x;
  const float r1 = (x == -INFINITY) ? 0.0f : x - (float)h;
  m = (__bf16)r1;
  l = (__bf16)(r1 - (float)m);
}

// c times the 8 bf16 values of v as three bf16 vectors.
__device__ __forceinline__ void split3_scaled(const uint4& v, float c, uint4& hi, uint4& mid, uint4& lo) {
  const bf16x8 x = __builtin_bit_cast(bf16x8, v);
  bf16x8 h, m, l;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    __bf16 a, b, d;
    split3((float)x[i] * c, a, b, d);
    h[i] = a;
    m[i] = b;
    l[i] = d;
  }
  hi = __builtin_bit_cast(uint4, h);
  mid = __builtin_bit_cast(uint4, m);
  lo = __builtin_bit_cast(uint4, l);
}

// Head dim 8, N a multiple of 32 (XP): the score product yields the
// exponent itself (the mask of a partial last key block would need more
// registers than four waves per SIMD leave). The key
// rows hold c k (c = scale log2 e) as three bf16 terms in features 0..23 and
// ones in 24..26; the lane's query operand holds q against each of the
// three terms and -r (r: the lane's reference, three bf16 terms) against the
// ones; the accumulator starts from bias log2 e. So x = bias log2 e +
// c q.k - r needs no vector work before its exp2. The value rows hold a
// one in feature 8, so the P V product also accumulates the row sum of P.
// The reference is kept 7 above the largest exponent seen when it is set,
// so every P of a block is below 2 unless some exponent has risen 8 or more
// above the row max: a bit test on the packed bf16 P finds that (or a
// non-finite P) and takes the exact path, which moves the reference and
// rescales the accumulators (row sum included) and the already issued
// scores of the next block.
constexpr float kRefHeadroom = 7.0f;

// p = 2^x as bf16, four at a time (the scheduling fences keep the fp32
// values from being held all at once beside x, which stays live for the
// exact path).
__device__ __forceinline__ void exp_only(const float (&x)[16], bf16x8& p0, bf16x8& p1) {
#pragma unroll
  for (int r = 0; r < 16; r += 4) {
    const float e0 = exp2_fast(x[r]), e1 = exp2_fast(x[r + 1]);
    const float e2 = exp2_fast(x[r + 2]), e3 = exp2_fast(x[r + 3]);
    bf16x8& d = r < 8 ? p0 : p1;
    d[r & 7] = (__bf16)e0;
    d[(r & 7) + 1] = (__bf16)e1;
    d[(r & 7) + 2] = (__bf16)e2;
    d[(r & 7) + 3] = (__bf16)e3;
    sched_fence();
  }
}

template <int D>
__device__ __forceinline__ void softmax_pv_xp(const f32x16& s, f32x16& sn, const bf16x8 (&vop)[2][D / 32],
                                              SoftmaxState& st, bf16x8& qm, f32x16 (&acc)[D / 32]) {
  constexpr int NCB = D / 32;
  const int g = (threadIdx.x >> 5) & 1;
  float x[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) x[r] = s[r];
  bf16x8 p0, p1;
  exp_only(x, p0, p1);
  const uint4 u0 = __builtin_bit_cast(uint4, p0), u1 = __builtin_bit_cast(uint4, p1);
  const uint32_t any_big = (u0.x | u0.y | u0.z | u0.w | u1.x | u1.y | u1.z | u1.w) & 0x40004000u;
  if (__any(any_big != 0u || st.m == -INFINITY)) {
    // x holds exponents relative to the old reference (absolute while there
    // is none, mneg = 0)
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, x[r]);
    mx -= st.mneg;
    const float mall = fmaxf(mx, __shfl_xor(mx, 32));
    const float mnew = fmaxf(st.m, mall + kRefHeadroom);
    const float alpha = (mnew == -INFINITY) ? 1.0f : exp2_fast(st.m - mnew);
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[cb][r] *= alpha;
    const float mneg_new = (mnew == -INFINITY) ? 0.0f : -mnew;
    const float shift = mneg_new - st.mneg;
    st.m = mnew;
    st.mneg = mneg_new;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      x[r] += shift;
      sn[r] += shift;
    }
    if (g == 1) {
      __bf16 h, m, l;
      split3(mneg_new, h, m, l);
      qm = zero_bf16x8();
      qm[0] = h;
      qm[1] = m;
      qm[2] = l;
    }
    exp_only(x, p0, p1);
  }
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    acc[cb] = mfma32(vop[0][cb], p0, acc[cb]);
    acc[cb] = mfma32(vop[1][cb], p1, acc[cb]);
  }
}

// XP, the first key block of a sequence (no reference yet, acc = 0): the
// reference is set from the block's maxima before the one exp2, and the
// next block's scores, issued without a reference, are moved to it.
template <int D>
__device__ __forceinline__ void softmax_first_xp(const f32x16& s, f32x16& sn, const bf16x8 (&vop)[2][D / 32],
                                                 SoftmaxState& st, bf16x8& qm, f32x16 (&acc)[D / 32]) {
  constexpr int NCB = D / 32;
  const int g = (threadIdx.x >> 5) & 1;
  float mx = -INFINITY;
#pragma unroll
  for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[r]);
  const float mall = fmaxf(mx, __shfl_xor(mx, 32));
  st.m = mall + kRefHeadroom;                       // -inf stays -inf
  st.mneg = (st.m == -INFINITY) ? 0.0f : -st.m;
  float x[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    x[r] = s[r] + st.mneg;
    sn[r] += st.mneg;
  }
  if (g == 1) {
    __bf16 h, m, l;
    split3(st.mneg, h, m, l);
    qm = zero_bf16x8();
    qm[0] = h;
    qm[1] = m;
    qm[2] = l;
  }
  bf16x8 p0, p1;
  exp_only(x, p0, p1);
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    acc[cb] = mfma32(vop[0][cb], p0, acc[cb]);
    acc[cb] = mfma32(vop[1][cb], p1, acc[cb]);
  }
}

// The first key block of a sequence on the FMA path (no reference yet,
// acc = 0, l = 0): the reference is set to the block's row max before the
// one exp2, as the exact path of softmax_pv would after a first exp2.
template <int D>
__device__ __forceinline__ void softmax_first(const f32x16& s, const bf16x8 (&vop)[2][D / 32], float sl2,
                                              SoftmaxState& st, f32x16 (&acc)[D / 32]) {
  constexpr int NCB = D / 32;
  float x[16];
  float mx = -INFINITY;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    x[r] = s[r] * sl2;
    mx = fmaxf(mx, x[r]);
  }
  const float mall = fmaxf(mx, __shfl_xor(mx, 32));
  st.m = mall;
  st.mneg = (mall == -INFINITY) ? 0.0f : -mall;
#pragma unroll
  for (int r = 0; r < 16; ++r) x[r] += st.mneg;
  bf16x8 p0, p1;
  st.l = exp_block(x, p0, p1);
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    acc[cb] = mfma32(vop[0][cb], p0, acc[cb]);
    acc[cb] = mfma32(vop[1][cb], p1, acc[cb]);
  }
}

// Persistent forward for sequences of at most 256 rows, N a multiple of 4,
// with at most 127 buckets (bf16 in and out, head dims 8, 16, 32 on 32-wide
// tiles; spd rows 4-byte aligned). Each wave owns 32 queries, and the
// sequence's K and V (all rows) sit in LDS: one pair of barriers per
// sequence instead of one barrier per key tile. At N > 128 a workgroup
// covers one sequence; shorter ones are packed, 2, 4 or 8 sequences of the
// head at once (N <= 128, 64, 32), each in its own slice of the K and V
// rows with 4, 2 or 1 waves. The per-lane bias table holds the byte values
// 0..127 (bytes of 128 or more are mapped to the padding entry 127, bias 0)
// and an entry of -inf (128) that masks the keys past N: with K and V that
// is about 71 KB, so two workgroups share a compute unit and every SIMD
// runs four waves. The workgroups are persistent: workgroup w takes head
// (w mod hpb) of every (G / hpb)-th group of sequences, fills the table
// once, and loads the next group's K, V and Q rows into registers while it
// computes the current one. spd words stream two key blocks ahead across
// groups (read 16 bytes at a time from 4-byte aligned offsets, through a
// resource that ends with the sequence's matrix); the score product of key
// block kb + 1 is issued before the softmax of block kb. TAIL: keys past N
// in the last block (N not a multiple of 32, or N <= 32).
constexpr int kShortTabEntries = 129;
template <int DS, bool TAIL>
__global__ __launch_bounds__(kThreads, DS <= 16 ? 4 : 2) void fwd_short_bf16_kernel(FwdArgs a) {
  constexpr int D = 32;
  constexpr int NKC = D / 16;
  constexpr int NKS = (DS + 15) / 16;
  constexpr int NCB = D / 32;
  constexpr int ROWS = 256;
  constexpr int CPS = DS / 8;                   // 16-byte chunks per source row
  constexpr int PER = ROWS * CPS;               // chunks per tensor (a multiple of 64)
  constexpr int IPT = (PER + kThreads - 1) / kThreads;
  constexpr bool XP = DS == 8 && !TAIL;         // exponents from the score product
  constexpr int NKP = XP ? 2 : NKS;             // 16-feature chunks of the score product
  // alternating score sets where registers allow: at d = 32 (one workgroup
  // per compute unit) and at d = 8 without a partial key block; elsewhere
  // the copy keeps four waves per SIMD without spilling
  constexpr bool ALT = DS == 32 || XP;
  // Padding rows (zero): the K rows of block nkb mod 8, read past the last
  // block of a sequence (the product is never used), and at N <= 32 the K
  // and V rows of the masked second block of the last slice stay in the
  // arrays (their P is 0, and the V rows must be finite)
  constexpr int KROWS = ROWS + 64, VROWS = ROWS + 32;
  __shared__ __attribute__((aligned(16))) uint16_t sK[KROWS * D], sV[VROWS * D];
  __shared__ __attribute__((aligned(16))) float sTab[kShortTabEntries * 64];

  const int tid = threadIdx.x;
  const int lane = tid & 63, w = wave_id();
  const int col = lane & 31, g = lane >> 5;
  const uint32_t lane4 = (uint32_t)lane * 4u;
  const int N = (int)a.Sq;
  // key blocks: at least 2 (N <= 32 has a second block whose keys are all
  // masked, so the spd stream below needs no case of its own)
  const int nkb = N > 32 ? (N + 31) / 32 : 2;
  // P sequences of the head at once (N <= 128: 2, N <= 64: 4, N <= 32: 8):
  // sequence slot p = w / GW of a group holds LDS rows p R .. p R + R - 1
  // and its waves take query blocks wl = w mod GW.
  const int lgp = N > 128 ? 0 : (N > 64 ? 1 : (N > 32 ? 2 : 3));
  const int P = 1 << lgp, GW = kWaves >> lgp, R = ROWS >> lgp;
  const int p = w >> (3 - lgp), wl = w & (GW - 1);
  const int G = (int)gridDim.x;
  const int lw = (int)xcd_remap(blockIdx.x, G);
  const int head = lw % a.hpb;
  const int slot = lw / a.hpb;
  const int nslots = G / a.hpb;
  const int nseq = a.H / a.hpb;
  const int ngroups = (nseq + P - 1) >> lgp;
  const float sl2 = a.scale * kLog2e;
  const int ld = (int)a.ld_spd;
  const int qi = wl * 32 + col;                 // this lane's query (in its sequence)
  const int qc = qi < N ? qi : N - 1;
  const bool wrows = wl * 32 < N;               // the wave owns query rows
  const uint16_t* sKp = sK + p * R * D;         // this wave's slice of K and V
  const uint16_t* sVp = sV + p * R * D;
  const FwdOffsets<D> off;

  // table entry (b, lane) at float 64 b + lane: bias / scale (XP: bias
  // log2 e) for b below n_buckets, 0 up to 127, -inf at 128; zero K, V
  // (features past the head dim stay zero; XP: the ones of feature 24..26
  // of K and feature 8 of V)
  {
    const float tmul = XP ? kLog2e : 1.0f / a.scale;
    const float* th = a.table + (int64_t)head * a.n_buckets;
    for (int t = tid; t < kShortTabEntries * 16; t += kThreads) {
      const int bk = t >> 4;
      const float x = bk < 128 ? (bk < a.n_buckets ? th[bk] * tmul : 0.0f) : -INFINITY;
      reinterpret_cast<float4*>(sTab)[t] = make_float4(x, x, x, x);
    }
    constexpr uint32_t kOne = 0x3f80u;           // bf16 1.0
    for (int t = tid; t < KROWS * D / 8; t += kThreads) {
      const int row = t >> 2, ch = t & 3;
      const int lo = row * D + swz_tile<D>(row, ch) * 8;
      const bool k1 = XP && ch == 3, v1 = XP && ch == 1;
      *reinterpret_cast<uint4*>(sK + lo) = make_uint4(k1 ? kOne | (kOne << 16) : 0u, k1 ? kOne : 0u, 0u, 0u);
      if (row < VROWS) *reinterpret_cast<uint4*>(sV + lo) = make_uint4(v1 ? kOne : 0u, 0u, 0u, 0u);
    }
  }

  // The wave's sequence in group gi (clamped to the batch for loads).
  auto seq_of = [&](int gi) { return (gi << lgp) + p; };
  auto clamp_seq = [&](int s) { return s < nseq ? s : nseq - 1; };
  // Loads of group gi into registers: its K and V rows (item u = row *
  // DS/8 + chunk, thread u mod 512; row r is row r mod R of the group's
  // sequence r / R; rows past N or past the batch read zero) and this lane's
  // Q row.
  uint4 rk[IPT], rv[IPT];
  bf16x8 qf[NKC], qn[XP ? 1 : NKC];
  auto issue = [&](int gi) {
    // resources from the group's first sequence (this head) to the end of
    // the tensors; the P sequences' rows are hpb N DS elements apart
    const int64_t base = ((int64_t)(gi << lgp) * a.hpb + head) * N * DS;
    const int64_t left = ((int64_t)a.H * N * DS - base) * 2;
    const int64_t nbytes = left < (int64_t)kZeroChunk ? left : (int64_t)kZeroChunk;
    const __amdgpu_buffer_rsrc_t sk = make_rsrc_n(reinterpret_cast<const uint16_t*>(a.k) + base, nbytes);
    const __amdgpu_buffer_rsrc_t sv = make_rsrc_n(reinterpret_cast<const uint16_t*>(a.v) + base, nbytes);
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int u = tid + i * kThreads;
      if (u < PER) {
        const int r = u / CPS, pr = r / R, lr = r - pr * R;
        const bool ok = lr < N && (gi << lgp) + pr < nseq;
        const uint32_t vo = ok ? (uint32_t)(((pr * a.hpb) * N + lr) * DS * 2 + (u % CPS) * 16) : kZeroChunk;
        rk[i] = buf_b128(sk, vo);
        rv[i] = buf_b128(sv, vo);
      }
    }
    const int h = clamp_seq(seq_of(gi)) * a.hpb + head;
    const uint16_t* qh = reinterpret_cast<const uint16_t*>(a.q) + (int64_t)h * N * DS;
    if constexpr (XP) {
      // the q row (the second operand is formed from it when the sequence starts)
      qn[0] = *reinterpret_cast<const bf16x8*>(qh + (int64_t)qc * DS);
    } else {
#pragma unroll
      for (int kc = 0; kc < NKC; ++kc)
        qn[kc] = (kc * 16 + g * 8 < DS) ? *reinterpret_cast<const bf16x8*>(qh + (int64_t)qc * DS + kc * 16 + g * 8)
                                        : zero_bf16x8();
    }
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

  // One group: its K, V, Q are in registers on entry (loaded during the
  // previous one), and wd[0], wd[1] hold the first spd words of the wave's
  // sequence. The spd words stream over (group, key block) two blocks ahead:
  // past the last block come blocks 0 and 1 of the wave's sequence in the
  // next group.
  auto run = [&](int gi) {
    const int s = seq_of(gi);
    const bool wact = wrows && s < nseq;
    const int gnx = gi + nslots < ngroups ? gi + nslots : gi;
    const __amdgpu_buffer_rsrc_t rs = spd_rs(clamp_seq(s));
    const __amdgpu_buffer_rsrc_t rn = spd_rs(clamp_seq(seq_of(gnx)));
    __syncthreads();            // the previous group's reads of K and V are done
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int u = tid + i * kThreads;
      if (u < PER) {
        const int row = u / CPS, chunk = u % CPS;
        const int lo = row * D + swz_tile<D>(row, chunk) * 8;
        if constexpr (XP) {
          uint4 hi, mid, low;
          split3_scaled(rk[i], sl2, hi, mid, low);
          *reinterpret_cast<uint4*>(sK + lo) = hi;
          *reinterpret_cast<uint4*>(sK + row * D + swz_tile<D>(row, 1) * 8) = mid;
          *reinterpret_cast<uint4*>(sK + row * D + swz_tile<D>(row, 2) * 8) = low;
        } else {
          *reinterpret_cast<uint4*>(sK + lo) = rk[i];
        }
        *reinterpret_cast<uint4*>(sV + lo) = rv[i];
      }
    }
    if constexpr (XP) {
      // q against the three key terms; zero against the ones (no reference yet)
      qf[0] = qn[0];
      qf[1] = g == 0 ? qn[0] : zero_bf16x8();
    } else {
#pragma unroll
      for (int kc = 0; kc < NKC; ++kc) qf[kc] = qn[kc];
    }
    __syncthreads();            // K, V of this group visible
    issue(gnx);
    sched_fence();
    st.m = -INFINITY;
    st.mneg = 0.0f;
    st.l = 0.0f;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[cb] = zero_f32x16();
    // Key block kb: the words of block kb + 2 are fetched (of the next
    // sequence past the end: one load whatever the source, so the wait for
    // block kb + 1's words leaves it in flight), block kb + 1's scores go
    // into sn (also past the last block: rows of the slice, of the next
    // slice or of the padding, and the result is never read),
    // and block kb's scores sc are softmaxed into acc.
    auto block = [&](int kb, f32x16& sc, f32x16& sn) {
      {
        const int kf = kb + 2;
        const bool here = kf < nkb;
        const __amdgpu_buffer_rsrc_t src = here ? rs : rn;
        buf_u128(src, voff, (uint32_t)((here ? kf : kf - nkb) * 32), wd[(kb + 2) % 3]);
      }
      sched_fence();
      if (wact) {
        {
          uint32_t e[4];
          entries(wd[(kb + 1) % 3], kb + 1, e);
          issue_scores<D, NKP>(sTab, e, lane4, sKp, off.k, (kb + 1) & 7, qf, sn);
        }
        bf16x8 vop[2][NCB];
        read_v<D>(sVp, off, kb, vop);
        if constexpr (XP) {
          if (kb == 0)
            softmax_first_xp<D>(sc, sn, vop, st, qf[1], acc);
          else
            softmax_pv_xp<D>(sc, sn, vop, st, qf[1], acc);
        } else {
          if (kb == 0)
            softmax_first<D>(sc, vop, sl2, st, acc);
          else
            softmax_pv<D, false>(sc, vop, 32, sl2, st, acc);
        }
        if constexpr (!ALT) sc = sn;
      }
    };
    if constexpr (ALT) {
      // the score sets of the even and odd blocks alternate, so neither is
      // copied (the break keeps a softmaxed set from being live afterwards)
      f32x16 sa, sb;
      if (wact) {
        uint32_t e[4];
        entries(wd[0], 0, e);
        issue_scores<D, NKP>(sTab, e, lane4, sKp, off.k, 0, qf, sa);
      }
#pragma unroll
      for (int kb = 0; kb < ROWS / 32; ++kb) {
        if (kb >= nkb) break;
        if (kb & 1)
          block(kb, sb, sa);
        else
          block(kb, sa, sb);
      }
    } else {
      f32x16 sc;
      if (wact) {
        uint32_t e[4];
        entries(wd[0], 0, e);
        issue_scores<D, NKP>(sTab, e, lane4, sKp, off.k, 0, qf, sc);
      }
#pragma unroll
      for (int kb = 0; kb < ROWS / 32; ++kb) {
        if (kb < nkb) {
          f32x16 sn;
          block(kb, sc, sn);
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
      // XP: the row sum is O^T row 8, register 4 of the lane half g = 0
      const float lt = XP ? __shfl(acc[0][4], col) : st.l + __shfl_xor(st.l, 32);
      if (qi < N) {
        // stores through resources over this head's rows (scalar bases,
        // 32-bit lane offsets: no 64-bit address is kept across sequences)
        const int h = s * a.hpb + head;   // s < nseq here
        const float inv = lt > 0.0f ? 1.0f / lt : 0.0f;
        const float lse_out = lt > 0.0f ? (st.m + __log2f(lt)) * kLn2 : -INFINITY;
        const __amdgpu_buffer_rsrc_t ro =
            make_rsrc_n(reinterpret_cast<uint16_t*>(a.o) + (int64_t)h * N * DS, (int64_t)N * DS * 2);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int c = 8 * u + 4 * g;
          if (c >= DS) continue;
          u32x2 pk;
          pk[0] = (uint32_t)f2bf(acc[0][4 * u] * inv) | ((uint32_t)f2bf(acc[0][4 * u + 1] * inv) << 16);
          pk[1] = (uint32_t)f2bf(acc[0][4 * u + 2] * inv) | ((uint32_t)f2bf(acc[0][4 * u + 3] * inv) << 16);
          __builtin_amdgcn_raw_buffer_store_b64(pk, ro, (uint32_t)((qi * DS + c) * 2), 0, 0);
        }
        if (g == 0) {
          const __amdgpu_buffer_rsrc_t rl = make_rsrc_n(a.lse + (int64_t)h * N, (int64_t)N * 4);
          __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(lse_out), rl, (uint32_t)(qi * 4), 0, 0);
        }
      }
    }
  };

  issue(slot);
  {
    const __amdgpu_buffer_rsrc_t rs = spd_rs(clamp_seq(seq_of(slot)));
    buf_u128(rs, voff, 0u, wd[0]);
    buf_u128(rs, voff, 32u, wd[1]);
  }
  for (int gi = slot; gi < ngroups; gi += nslots) run(gi);
  wait_vmcnt<0>();     // drain the loads issued for the last (repeated) sequence
}

template <int DS>
void launch_short_t(const FwdArgs& a, hipStream_t s) {
  const int nseq = a.H / a.hpb;
  const int lgp = a.Sq > 128 ? 0 : (a.Sq > 64 ? 1 : (a.Sq > 32 ? 2 : 3));   // 2^lgp sequences per workgroup
  const int ngroups = (nseq + (1 << lgp) - 1) >> lgp;
  // two workgroups per compute unit where the registers allow four waves per SIMD
  int slots = (DS <= 16 ? 512 : 256) / a.hpb;
  if (slots < 1) slots = 1;
  if (slots > ngroups) slots = ngroups;
  const dim3 grid((unsigned)(slots * a.hpb));
  if (a.Sq % 32 != 0 || a.Sq <= 32)   // keys past N masked (at N <= 32 the whole second block)
    hipLaunchKernelGGL((fwd_short_bf16_kernel<DS, true>), grid, dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((fwd_short_bf16_kernel<DS, false>), grid, dim3(kThreads), 0, s, a);
}

}  // namespace

bool fwd_short_applies(const FwdArgs& a, int d) {
  // (a group of up to 8 sequences is read through one resource of at most
  // 2^30 bytes)
  return d <= 32 && !a.accumulate && a.row_off == 0 && a.col_off == 0 && a.Sq == a.Sk &&
         a.Sq >= 1 && a.Sq <= 256 && a.Sq % 4 == 0 &&   // (keys past N are masked by spd words)
         a.n_buckets <= 127 && a.hpb >= 1 && a.H % a.hpb == 0 &&
         (int64_t)8 * a.hpb * a.Sq * d * 2 < ((int64_t)1 << 30) &&
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
