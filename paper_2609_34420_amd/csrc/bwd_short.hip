// Backward for sequences of at most 256 rows (bf16, head dims 8, 16, 32):
// dK, dV, dQ and the bias-table gradient in one kernel.
//
// One workgroup of 8 waves covers every key of a sequence (wave w owns keys
// 32 w .. 32 w + 31, lane & 31 = key), so each 32 x 32 block of scores is
// formed once. P and dS feed dV^T += dO^T P and dK^T += Q^T dS straight from
// registers, as in the key-stationary kernel, and dQ = scale dS K is reduced
// inside the workgroup instead of by a second pass that recomputes S and dP.
// The 8 x 8 blocks are visited on diagonals: at step t wave w forms block
// (query block (w + t) mod 8, key block w) and stores its dS (bf16) in an LDS
// slot; after the step's barrier wave w adds to dQ of its own query block w
// the block (w, (w - t) mod 8), stored by wave (w - t) mod 8 at that step,
// as dQ^T += K^T dS^T with both operands read by transposing LDS reads. So
// every wave accumulates dK and dV of its key block and dQ of its query block
// in registers across the 8 steps, and every stored block is read by one
// wave. The slots are double buffered by step parity.
//
// Shorter sequences are packed: at N <= 128 (64, 32) a workgroup takes 2
// (4, 8) sequences of its head at once, each in its own slice of the LDS
// rows with 4 (2, 1) waves that run the same diagonal schedule over 4 (2, 1)
// blocks, so no wave waits through steps that hold no block of its sequence.
//
// The workgroups are persistent: there are at most 256 of them (one per
// compute unit, the kernel holds 160 KiB of LDS) and workgroup w takes head
// (w mod hpb) of every (G / hpb)-th group of sequences, G the grid size. Its bias table
// and gradient histogram (the key-stationary kernel's layout and fixed-point
// scheme) stay in LDS across its sequences: the table is filled and the
// histogram flushed once. The histogram's power-of-two scale follows the
// largest norm bound seen so far (it only decreases; the accumulated sums are
// shifted when it does). A group's loads are issued during the last step
// of the one before. The hpb heads of a sequence run on one XCD at about the
// same time, so they share its spd bytes in L2.
//
// The prepare stage's work is done here too: each sequence's Dlt = rowsum(dO * O),
// LSE log2 e and norm maxima come from its rows as they are loaded.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "stage.hpp"

namespace gt {

namespace {

constexpr int kNW = 8;               // waves per workgroup
constexpr int kThreads = kNW * 64;
constexpr int kRows = 256;           // longest sequence: 8 blocks of 32 rows
constexpr int D = 32;                // tile width; head dims below it are zero-padded
constexpr uint32_t kTabBase = 65536;
constexpr int kMaxGridShort = 256;

template <int NB>
constexpr int copies() { return NB <= 128 ? 32 : 16; }

// LDS below 64 KiB: the sequence's Q, dO and K rows (row-major, the tile
// swizzle of 64-row tiles, rows past N and features past the head dim zero),
// the accumulator starts of S and dP per query, and -inf starts for the
// lanes of keys past N.
struct ShortTiles {
  uint16_t q[kRows * D];
  uint16_t o[kRows * D];
  uint16_t k[kRows * D];
  float init_s[kRows];                // -LSE log2 e / (scale log2 e); -inf past N
  float init_p[kRows];                // -Dlt 2^F
  float ninf[kRows];                  // -inf: S start of the keys past N, so P = 0
  float red[3][kNW];
};
// From 64 KiB: table copies, histogram copies (as in the key-stationary
// kernel: the histogram entry at a fixed offset from the table entry), then
// the dS slots: [step parity][writer wave], 32 keys (rows) x 32 queries in
// the 32-wide tile layout.
template <int NB>
struct ShortSmem : ShortTiles {
  static constexpr int ENT = NB * copies<NB>();
  uint8_t pad[kTabBase - sizeof(ShortTiles)];
  uint2 tabw[ENT];
  unsigned long long hist[ENT];
  uint16_t xs[2][kNW][32 * D];
};
static_assert(sizeof(ShortSmem<128>) <= 160 * 1024 && sizeof(ShortSmem<256>) <= 160 * 1024,
              "LDS budget");

__device__ __forceinline__ int round_to_int(float x) {
  int r;
  asm("v_cvt_rpi_i32_f32 %0, %1" : "=v"(r) : "v"(x));   // floor(x + 0.5)
  return r;
}

// Byte values of 128 and more have no entry in the 128-bucket layout, which
// is used only when n_buckets <= 127: they are mapped to its padding bucket
// 127 (bias 0, gradient discarded). Valid input never takes the branch.
template <int NB>
__device__ __forceinline__ void clamp_buckets(uint32_t (&w)[4]) {
  if constexpr (NB <= 128) {
    if (__any(((w[0] | w[1] | w[2] | w[3]) & 0x80808080u) != 0)) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        uint32_t x = w[u];
#pragma unroll
        for (int k = 0; k < 4; ++k)
          if ((x >> (8 * k + 7)) & 1u) x = (x & ~(0xffu << (8 * k))) | (0x7fu << (8 * k));
        w[u] = x;
      }
    }
  }
}
// Per-lane LDS element offsets of the operand reads.
struct ShortOffsets {
  int row[D / 16];     // rows perm32(lane) of a 32-row block, feature chunk 2 kc + g
  int tr[2];           // transposing reads h = 0, 1 (tile columns 0..31)
  __device__ __forceinline__ ShortOffsets() {
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) row[kc] = row_operand_off<D>(kc);
#pragma unroll
    for (int h = 0; h < 2; ++h) tr[h] = tr_operand_off<D>(h, 0);
  }
};

// Block (query block qb, this wave's keys): S and dP, P and dS, the bias
// reads and gradient adds, dV and dK, and dS (bf16) into slot xs.
// b: the lane's 16 bucket indices (4 words of spd_t, or 16 gathered bytes).
// SPROD: the statistics come with the products (features DS..DS+2 of the Q
// and dO rows hold -LSE / scale and -Dlt, and the lane's K and V operands
// ones and 2^F there; NKS then counts the chunk that holds them), so S and dP
// start from zero.
// rb: first LDS row of the wave's sequence (its slice when several
// sequences share the workgroup).
template <int NKS, int NB, bool SPROD, typename BT>
__device__ __forceinline__ void block_dkdv(ShortSmem<NB>& sm, const ShortOffsets& off,
                                           const bf16x8* kf, const bf16x8* vf, const BT* b,
                                           const float* is_lane, float sl2, int rb, int qb, uint16_t* xs,
                                           f32x16& dk, f32x16& dv) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 5;
  const int ib = rb + qb * 32 + 16 * g;   // this lane half's first query (LDS row)

  f32x16 s, dp;
  if constexpr (SPROD) {
    s = zero_f32x16();
    dp = zero_f32x16();
  } else {
    const float4* is4 = reinterpret_cast<const float4*>(is_lane + rb + qb * 32);
    const float4* ip4 = reinterpret_cast<const float4*>(&sm.init_p[ib]);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float4 x = is4[u], y = ip4[u];
      s[4 * u] = x.x; s[4 * u + 1] = x.y; s[4 * u + 2] = x.z; s[4 * u + 3] = x.w;
      dp[4 * u] = y.x; dp[4 * u + 1] = y.y; dp[4 * u + 2] = y.z; dp[4 * u + 3] = y.w;
    }
  }
#pragma unroll
  for (int kc = 0; kc < NKS; ++kc) {
    s = mfma32(lds_b128(sm.q + (rb + qb * 32) * D + off.row[kc]), kf[kc], s);
    dp = mfma32(lds_b128(sm.o + (rb + qb * 32) * D + off.row[kc]), vf[kc], dp);
  }
  float p[16], ds[16];
  uint32_t addr[16];   // LDS byte offset of table entry (bucket, copy) from sm
  float tb[16];
  constexpr int CPY = copies<NB>();
  const uint32_t cpyb = (uint32_t)(lane & (CPY - 1)) * 8u | kTabBase;
  uint32_t w[4];
  if constexpr (sizeof(BT) == 4) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      w[u] = b[u];
      opaque(w[u]);
    }
  } else {
    // 16 gathered bytes (one per register, upper bits unknown to the
    // compiler) packed into 4 words by byte permutes
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      uint32_t x[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        x[e] = b[4 * u + e];
        opaque(x[e]);
      }
      const uint32_t lo = __builtin_amdgcn_perm(x[1], x[0], 0x0c0c0400u);
      const uint32_t hi = __builtin_amdgcn_perm(x[3], x[2], 0x0c0c0400u);
      w[u] = __builtin_amdgcn_perm(hi, lo, 0x05040100u);
    }
  }
  clamp_buckets<NB>(w);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    if constexpr (CPY == 32)
      addr[r] = __builtin_amdgcn_perm(w[r >> 2], cpyb, 0x0c020000u | ((4u + (r & 3)) << 8));
    else
      addr[r] = (((w[r >> 2] >> (8 * (r & 3))) & 0xffu) << 7) | cpyb;
  }
  const uint8_t* lds0 = reinterpret_cast<const uint8_t*>(&sm);
#pragma unroll
  for (int r = 0; r < 16; ++r) tb[r] = *reinterpret_cast<const float*>(lds0 + addr[r]);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const float pv = exp2_fast(fmaf(s[r], sl2, tb[r]));
    p[r] = pv;
    ds[r] = pv * dp[r];
  }
  constexpr uint32_t kHistOff = ShortSmem<NB>::ENT * 8;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    unsigned long long* hp =
        reinterpret_cast<unsigned long long*>(const_cast<uint8_t*>(lds0) + addr[r] + kHistOff);
    atomicAdd(hp, (unsigned long long)(long long)round_to_int(ds[r]));
  }
  const int key = lane & 31;
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const bf16x8 pb = cvt_bf16x8(p + 8 * q);
    const bf16x8 db = cvt_bf16x8(ds + 8 * q);
    const int base = (rb + qb * 32 + 8 * q) * D;
    dv = mfma32(lds_tr_operand(sm.o + base, off.tr[0], off.tr[1]), pb, dv);
    dk = mfma32(lds_tr_operand(sm.q + base, off.tr[0], off.tr[1]), db, dk);
    // queries 16 g + 8 q .. + 7 of this key: chunk 2 g + q of slot row `key`
    *reinterpret_cast<bf16x8*>(xs + key * D + swz_tile<D>(key, 2 * g + q) * 8) = db;
  }
}

// STAGE (no transpose given, spd rows 4-byte aligned): the spd block of a
// step is loaded row-wise, 16 bytes per lane (lane l: row l / 2, bytes
// 16 (l % 2) .. + 15 of the block's 32 x 32), written to the first KiB of
// the wave's dS slot of that step (free until the block's dS is stored
// there), and each lane reads its key's 16 query bytes back with two 8-bit
// transposing LDS reads, instead of 16 byte gathers from global memory.
// SPROD (head dims 8 and 16, N a multiple of 32): the S and dP accumulators
// start at zero, and -LSE / scale, -Dlt enter the products through the
// zero-padded features DS..DS+2 (three bf16 terms each, exact to about 2^-24)
// of the staged Q and dO rows against ones and 2^F in the lane's K and V
// operands, instead of eight LDS reads of statistics per block (at DS = 16
// one more 16-feature chunk of S and dP).
template <int DS, int NB, bool TR, bool STAGE, bool SPROD = false>
__global__ __launch_bounds__(kThreads, 1) void bwd_short_bf16_kernel(BwdArgs a) {
  constexpr int NKS = (DS + 15) / 16;   // 16-feature chunks of S and dP that hold data
  constexpr int CPS = DS / 8;           // 16-byte chunks per source row
  constexpr int CPY = copies<NB>();
  constexpr int PER = kRows * CPS;      // 16-byte items per tensor (a multiple of 64)
  constexpr int IPT = (PER + kThreads - 1) / kThreads;
  __shared__ __attribute__((aligned(16))) ShortSmem<NB> sm;
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int g = lane >> 5;
  const int w = wave_id();
  const int N = (int)a.Sq;
  const int nb = (N + 31) / 32;
  // P sequences of the head at once (N <= 128: 2, N <= 64: 4, N <= 32: 8):
  // sequence slot p = w / GW of a group holds LDS rows p R .. p R + R - 1,
  // and its GW waves run the diagonal schedule over GW blocks (wl = w mod
  // GW; one wave and one step at N <= 32).
  const int lgp = N > 128 ? 0 : (N > 64 ? 1 : (N > 32 ? 2 : 3));
  const int P = 1 << lgp, GW = kNW >> lgp, R = kRows >> lgp;
  const int p = w >> (3 - lgp), wl = w & (GW - 1);
  const int rb = p * R;

  const int G = (int)gridDim.x;
  const int lw = (int)xcd_remap(blockIdx.x, G);
  const int head = lw % a.hpb;
  const int slot = lw / a.hpb;
  const int nslots = G / a.hpb;
  const int nseq = a.H / a.hpb;
  const int ngroups = (nseq + P - 1) >> lgp;
  auto seq_of = [&](int gi) { return (gi << lgp) + p; };
  auto clamp_seq = [&](int s) { return s < nseq ? s : nseq - 1; };

  // Table (times log2 e) and histogram of this workgroup's head; zero tiles
  // (features past the head dim and rows past N stay zero); -inf starts.
  for (int t = tid; t < ShortSmem<NB>::ENT; t += kThreads) {
    const int bkt = t / CPY;
    const float tv = (bkt < a.n_buckets) ? a.table[(int64_t)head * a.n_buckets + bkt] * kLog2e : 0.0f;
    sm.tabw[t] = make_uint2(__float_as_uint(tv), 0u);
    sm.hist[t] = 0ull;
  }
  for (int t = tid; t < 3 * kRows * D / 8; t += kThreads)
    reinterpret_cast<uint4*>(sm.q)[t] = make_uint4(0u, 0u, 0u, 0u);
  for (int t = tid; t < kRows; t += kThreads) sm.ninf[t] = -INFINITY;

  const float sl2 = a.scale * kLog2e;
  const float inv_sl2 = 1.0f / sl2;
  const int key = lane & 31;
  const int j = wl * 32 + key;          // this lane's key (in its sequence)
  const bool jok = j < N;
  const int jc = jok ? j : N - 1;
  const float* is_lane = (jok ? sm.init_s : sm.ninf) + 16 * g;
  const ShortOffsets off;
  const int ld = (int)a.ld_spd;
  using BT = std::conditional_t<TR || STAGE, uint32_t, uint8_t>;
  constexpr int NBT = TR || STAGE ? 4 : 16;
  static_assert(!(TR && STAGE), "one way of reading spd");
  static_assert(!SPROD || DS <= 16, "statistics through the padded features need DS <= 16");
  constexpr int NKSP = SPROD ? (DS + 3 + 15) / 16 : NKS;   // chunks of S and dP with the statistics

  // The loads of a sequence, issued one sequence ahead (during the last step
  // of the previous one) into registers: its Q, dO, K and O rows, item u =
  // row * DS/8 + chunk held by thread u mod 512 (rows past N read zero: each
  // resource ends at row N), the LSE of the rows whose chunk 0 the thread
  // holds, and this lane's K and V row.
  uint4 rq[IPT], rd[IPT], rk[IPT], ro[IPT];
  float lsev[IPT], dltv[IPT];
  bf16x8 kraw[D / 16], vraw[D / 16];
  auto issue = [&](int gi) {
    // rows of the group through resources from its first sequence (this
    // head) to the end of the tensors (at most 2^30 bytes); the P sequences'
    // rows are hpb N DS elements apart, row r of the group is row r mod R of
    // its sequence r / R
    const int64_t base = ((int64_t)(gi << lgp) * a.hpb + head) * N * DS;
    const int64_t left = ((int64_t)a.H * N * DS - base) * 2;
    const int64_t nbytes = left < (int64_t)kZeroChunk ? left : (int64_t)kZeroChunk;
    const __amdgpu_buffer_rsrc_t sq = make_rsrc_n(reinterpret_cast<const uint16_t*>(a.q) + base, nbytes);
    const __amdgpu_buffer_rsrc_t sd = make_rsrc_n(reinterpret_cast<const uint16_t*>(a.d_o) + base, nbytes);
    const __amdgpu_buffer_rsrc_t sk = make_rsrc_n(reinterpret_cast<const uint16_t*>(a.k) + base, nbytes);
    const __amdgpu_buffer_rsrc_t so = make_rsrc_n(reinterpret_cast<const uint16_t*>(a.o) + base, nbytes);
    // Every load is issued (items past PER and features past the head dim
    // read zero past the resource's end; the LSE of a row past N is replaced
    // where it is used), so no loaded register merges with an older value
    // and none is copied, which would wait for the load.
    const int64_t lbase = (base / DS);
    const int64_t lleft = ((int64_t)a.H * N - lbase) * 4;
    const __amdgpu_buffer_rsrc_t sl =
        make_rsrc_n(a.lse + lbase, lleft < (int64_t)kZeroChunk ? lleft : (int64_t)kZeroChunk);
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int u = tid + i * kThreads;
      const int r = u / CPS, pr = r >> (8 - lgp), lr = r & (R - 1);
      const bool ok = u < PER && lr < N && (gi << lgp) + pr < nseq;
      const int prow = pr * a.hpb * N + lr;          // row in the resources
      const uint32_t voff = ok ? (uint32_t)(prow * DS * 2 + (u % CPS) * 16) : kZeroChunk;
      rq[i] = buf_b128(sq, voff);
      rd[i] = buf_b128(sd, voff);
      rk[i] = buf_b128(sk, voff);
      ro[i] = buf_b128(so, voff);
      lsev[i] = __uint_as_float(
          __builtin_amdgcn_raw_buffer_load_b32(sl, ok ? (uint32_t)(prow * 4) : kZeroChunk, 0, 0));
    }
    // this lane's key of the wave's sequence
    const int64_t wbase = ((int64_t)clamp_seq(seq_of(gi)) * a.hpb + head) * N * DS;
    const __amdgpu_buffer_rsrc_t sk1 = make_rsrc_n(reinterpret_cast<const uint16_t*>(a.k) + wbase, (int64_t)N * DS * 2);
    const __amdgpu_buffer_rsrc_t sv = make_rsrc_n(reinterpret_cast<const uint16_t*>(a.v) + wbase, (int64_t)N * DS * 2);
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) {
      const bool in = jok && kc * 16 + g * 8 < DS;
      // (out of range: moved past the end by kZeroChunk, without a branch)
      const uint32_t ko = (uint32_t)((jc * DS + kc * 16 + g * 8) * 2) + (in ? 0u : kZeroChunk);
      kraw[kc] = __builtin_bit_cast(bf16x8, buf_b128(sk1, ko));
      vraw[kc] = __builtin_bit_cast(bf16x8, buf_b128(sv, ko));
    }
  };
  // Statistics of the loaded sequence (the prepare stage's definitions and
  // order of operations): Dlt = dO . O and |dO|^2 per row, reduced over the
  // DS/8 lanes of the row; |V|^2 per key; their maxima per wave into red.
  auto stats = [&]() {
    // the loaded registers pass through an empty asm here, so no use of
    // them is moved ahead of this point (in particular into the last step,
    // where it would wait for loads meant to overlap that step)
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      opaque(ro[i]);
      opaque(rd[i]);
    }
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) {
      uint4 x = __builtin_bit_cast(uint4, vraw[kc]);
      opaque(x);
      vraw[kc] = __builtin_bit_cast(bf16x8, x);
    }
    float md = 0.0f, mv = 0.0f, ml = 0.0f;
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int u = tid + i * kThreads;
      if (u < PER) {
        const uint16_t* xp = reinterpret_cast<const uint16_t*>(&ro[i]);
        const uint16_t* yp = reinterpret_cast<const uint16_t*>(&rd[i]);
        float acc = 0.0f, sq = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float yf = bf2f(yp[e]);
          acc = fmaf(bf2f(xp[e]), yf, acc);
          sq = fmaf(yf, yf, sq);
        }
#pragma unroll
        for (int o = CPS / 2; o >= 1; o >>= 1) {
          acc += __shfl_xor(acc, o);
          sq += __shfl_xor(sq, o);
        }
        dltv[i] = acc;
        if (((u / CPS) & (R - 1)) < N) {     // rows past N (or of no sequence) hold zeros
          md = fmaxf(md, sq);
          ml = fmaxf(ml, fabsf(acc));
        }
      }
    }
    float vq = 0.0f;
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float x = (float)vraw[kc][e];
        vq = fmaf(x, x, vq);
      }
    vq += __shfl_xor(vq, 32);
    if (jok) mv = vq;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
      md = fmaxf(md, __shfl_xor(md, o));
      mv = fmaxf(mv, __shfl_xor(mv, o));
      ml = fmaxf(ml, __shfl_xor(ml, o));
    }
    if (lane == 0) {
      sm.red[0][w] = md;
      sm.red[1][w] = mv;
      sm.red[2][w] = ml;
    }
  };
  // spd bytes of block (qb, this wave's keys) of sequence s: rows
  // 32 qb + 16 g + r, column j (rows past N read zero).
  const uint32_t voff_st = (uint32_t)((lane >> 1) * ld + 16 * (lane & 1) + wl * 32);
  int off_tr8[2];   // byte offsets in the staged block of the two transposing reads
#pragma unroll
  for (int hh = 0; hh < 2; ++hh)
    off_tr8[hh] = (16 * g + 8 * hh + ((lane & 15) >> 1)) * 32 + 16 * ((lane >> 4) & 1) + 8 * (lane & 1);
  auto fetch = [&](int s, int qb, BT* dst) {
    const int h = s * a.hpb + head;
    const __amdgpu_buffer_rsrc_t rs =
        make_rsrc_n(TR ? seq_spd_t(a, h) : seq_spd(a, h), (int64_t)N * ld);
    if constexpr (STAGE) {
      buf_u128(rs, voff_st, (uint32_t)(qb * 32 * ld), reinterpret_cast<uint32_t*>(dst));
    } else if constexpr (TR) {
      buf_u128(rs, (uint32_t)(jc * ld + 16 * g), (uint32_t)(qb * 32), reinterpret_cast<uint32_t*>(dst));
    } else {
      const uint32_t voff = (uint32_t)((qb * 32 + 16 * g) * ld + jc);
#pragma unroll
      for (int r = 0; r < 16; ++r) dst[r] = (uint8_t)buf_u8(rs, voff, (uint32_t)(r * ld));
    }
  };

  // Fixed-point exponent F of the histogram: every term round(dS 2^F) stays
  // below 2^30 in magnitude, using |dS_ij| <= |dO_i| |V_j| + |Dlt_i| (P <= 1)
  // with the maxima of the sequences at hand. F only decreases; when it does,
  // the histogram accumulated so far is shifted to the new scale.
  int fexp = 40;
  bool used = false;

  BT bA[NBT], bB[NBT];
  issue(slot);
  fetch(clamp_seq(seq_of(slot)), wl, bA);
  stats();
  for (int gi = slot; gi < ngroups; gi += nslots) {
    const int seq = seq_of(gi);            // this wave's sequence (none if >= nseq)
    const int seqc = clamp_seq(seq);
    const int h = seqc * a.hpb + head;
    const int64_t rowbase = (int64_t)h * N * DS;
    // the previous group's readers are done with the tiles and slots, and
    // its histogram adds are complete
    lds_barrier();
    {
      float md = sm.red[0][0], mv = sm.red[1][0], ml = sm.red[2][0];
#pragma unroll
      for (int i = 1; i < kNW; ++i) {
        md = fmaxf(md, sm.red[0][i]);
        mv = fmaxf(mv, sm.red[1][i]);
        ml = fmaxf(ml, sm.red[2][i]);
      }
      // a 1.5 % margin covers the rounding of P and of the products
      const float bound = 1.015f * (sqrtf(md) * sqrtf(mv) + ml);
      int fs = 40;
      if (bound > 0.0f && bound < INFINITY) {
        int e;
        frexpf(bound, &e);                 // bound < 2^e
        fs = 30 - e;
        fs = fs > 40 ? 40 : (fs < -100 ? -100 : fs);
      }
      if (fs < fexp) {                     // workgroup-uniform
        if (used) {
          const int sh = fexp - fs > 63 ? 63 : fexp - fs;
          for (int t = tid; t < ShortSmem<NB>::ENT; t += kThreads)
            sm.hist[t] = (unsigned long long)((long long)sm.hist[t] >> sh);
        }
        fexp = fs;
      }
      used = true;
    }
    const float sF = ldexpf(1.0f, fexp);
    const float gscale = a.scale * ldexpf(1.0f, -fexp);   // dK and dQ: scale 2^-F
#pragma unroll
    for (int i = 0; i < IPT; ++i) {
      const int u = tid + i * kThreads;
      if (u < PER) {
        const int row = u / CPS, chunk = u % CPS;
        const int lo = row * D + swz_tile<D>(row, chunk) * 8;
        *reinterpret_cast<uint4*>(sm.q + lo) = rq[i];
        *reinterpret_cast<uint4*>(sm.o + lo) = rd[i];
        *reinterpret_cast<uint4*>(sm.k + lo) = rk[i];
        if (chunk == 0) {
          // S starts at -LSE log2 e / (scale log2 e) (-inf for an empty row
          // or a row past N, so P = 0), dP at -Dlt 2^F
          const bool rin = (row & (R - 1)) < N && (gi << lgp) + (row >> (8 - lgp)) < nseq;
          const float L = rin ? lsev[i] : -INFINITY;
          const float ss = (L == -INFINITY) ? -INFINITY : -(L * kLog2e) * inv_sl2;
          sm.init_s[row] = ss;
          sm.init_p[row] = rin ? -dltv[i] * sF : 0.0f;
          if constexpr (SPROD) {
            // features DS..DS+2 of the row: the start as three bf16 terms
            auto split3 = [](float x, uint4& c) {
              const float h = (float)(__bf16)x;
              const float r1 = (x == -INFINITY) ? 0.0f : x - h;
              const float m = (float)(__bf16)r1;
              const float l = r1 - m;
              c = make_uint4((uint32_t)f2bf(h) | ((uint32_t)f2bf(m) << 16), (uint32_t)f2bf(l), 0u, 0u);
            };
            uint4 cq, co;
            split3(ss, cq);
            split3(rin ? -dltv[i] : 0.0f, co);
            const int lo1 = row * D + swz_tile<D>(row, DS / 8) * 8;
            *reinterpret_cast<uint4*>(sm.q + lo1) = cq;
            *reinterpret_cast<uint4*>(sm.o + lo1) = co;
          }
        }
      }
    }
    // K and 2^F V of this lane's key as B operands (the scale is exact in bf16)
    bf16x8 kf[D / 16], vf[D / 16];
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) {
      kf[kc] = kraw[kc];
#pragma unroll
      for (int e = 0; e < 8; ++e) vf[kc][e] = (__bf16)((float)vraw[kc][e] * sF);
    }
    if constexpr (SPROD) {
      // features DS..DS+2 of the lane's K and V operands: chunk DS / 16,
      // lane half (DS / 8) & 1
      if (g == ((DS / 8) & 1) && jok) {
#pragma unroll
        for (int e = 0; e < 3; ++e) {
          kf[DS / 16][e] = (__bf16)1.0f;
          vf[DS / 16][e] = (__bf16)sF;
        }
      }
    }

    f32x16 dk = zero_f32x16(), dv = zero_f32x16(), dq = zero_f32x16();
    const bool wact = wl < nb && seq < nseq;
    auto step_a = [&](int t, uint16_t* xs, const BT* b) {
      const int qb = (wl + t) & (GW - 1);
      if (wact && qb < nb) {
        if constexpr (STAGE) {
          typedef int i32x2 __attribute__((ext_vector_type(2)));
          typedef __attribute__((address_space(3))) i32x2* lds_i32x2;
          uint8_t* st8 = reinterpret_cast<uint8_t*>(xs);
          uint4 v4 = make_uint4(b[0], b[1], b[2], b[3]);
          opaque(v4);
          *reinterpret_cast<uint4*>(st8 + 16 * lane) = v4;
          uint32_t wv[4];
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const i32x2 v = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2)(void*)(st8 + off_tr8[hh]));
            wv[2 * hh] = (uint32_t)v.x;
            wv[2 * hh + 1] = (uint32_t)v.y;
          }
          block_dkdv<NKSP, NB, SPROD>(sm, off, kf, vf, wv, is_lane, sl2, rb, qb, xs, dk, dv);
        } else {
          block_dkdv<NKSP, NB, SPROD>(sm, off, kf, vf, b, is_lane, sl2, rb, qb, xs, dk, dv);
        }
      }
    };
    auto step_b = [&](int t, int par) {
      const int src = (wl - t) & (GW - 1);   // key block whose dS for query block wl was stored at step t
      if (wact && src < nb) {
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          const bf16x8 kt = lds_tr_operand(sm.k + (rb + src * 32 + 8 * q) * D, off.tr[0], off.tr[1]);
          const bf16x8 sv = lds_tr_operand(&sm.xs[par][p * GW + src][8 * q * D], off.tr[0], off.tr[1]);
          dq = mfma32(kt, sv, dq);
        }
      }
    };

    wait_loads();
    lds_barrier();
#pragma unroll 1
    for (int t = 0; t < GW - 2; t += 2) {
      fetch(seqc, (wl + t + 1) & (GW - 1), bB);
      sched_fence();
      if (t > 0) step_b(t - 1, 1);
      step_a(t, sm.xs[0][w], bA);
      lds_barrier();
      fetch(seqc, (wl + t + 2) & (GW - 1), bA);
      sched_fence();
      step_b(t, 0);
      step_a(t + 1, sm.xs[1][w], bB);
      lds_barrier();
    }
    // The last two steps, with the next group's loads issued at the start
    // of the last one (the last group reloads itself, so the code is the
    // same on every path and the waits stay exact).
    // (GW = 1: only the last step, whose block is also in bB)
    fetch(seqc, (wl + GW - 1) & (GW - 1), bB);
    sched_fence();
    if (GW > 2) step_b(GW - 3, 1);
    if (GW > 1) step_a(GW - 2, sm.xs[0][w], bA);
    lds_barrier();
    {
      const int gnx = gi + nslots < ngroups ? gi + nslots : gi;
      issue(gnx);
      fetch(clamp_seq(seq_of(gnx)), wl, bA);
    }
    sched_fence();
    if (GW > 1) step_b(GW - 2, 0);
    step_a(GW - 1, sm.xs[1][w], bB);
    lds_barrier();
    step_b(GW - 1, 1);

    // dK, dV of key j; dQ of query j (features 8 u + 4 g .. + 3)
    if (jok && seq < nseq) {
      uint16_t* dkp = reinterpret_cast<uint16_t*>(a.dk) + rowbase + (int64_t)j * DS;
      uint16_t* dvp = reinterpret_cast<uint16_t*>(a.dv) + rowbase + (int64_t)j * DS;
      uint16_t* dqp = reinterpret_cast<uint16_t*>(a.dq) + rowbase + (int64_t)j * DS;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = 8 * u + 4 * g;
        if (c >= DS) continue;
        uint2 pk, pv, pq;
        pk.x = (uint32_t)f2bf(dk[4 * u] * gscale) | ((uint32_t)f2bf(dk[4 * u + 1] * gscale) << 16);
        pk.y = (uint32_t)f2bf(dk[4 * u + 2] * gscale) | ((uint32_t)f2bf(dk[4 * u + 3] * gscale) << 16);
        pv.x = (uint32_t)f2bf(dv[4 * u]) | ((uint32_t)f2bf(dv[4 * u + 1]) << 16);
        pv.y = (uint32_t)f2bf(dv[4 * u + 2]) | ((uint32_t)f2bf(dv[4 * u + 3]) << 16);
        pq.x = (uint32_t)f2bf(dq[4 * u] * gscale) | ((uint32_t)f2bf(dq[4 * u + 1] * gscale) << 16);
        pq.y = (uint32_t)f2bf(dq[4 * u + 2] * gscale) | ((uint32_t)f2bf(dq[4 * u + 3] * gscale) << 16);
        *reinterpret_cast<uint2*>(dkp + c) = pk;
        *reinterpret_cast<uint2*>(dvp + c) = pv;
        *reinterpret_cast<uint2*>(dqp + c) = pq;
      }
    }
    // statistics of the next sequence (its loads were issued above)
    stats();
  }
  lds_barrier();
  const double unscale = ldexp(1.0, -fexp);
  for (int bkt = tid; bkt < a.n_buckets; bkt += kThreads) {
    long long t = 0;
#pragma unroll
    for (int c = 0; c < CPY; ++c) t += (long long)sm.hist[bkt * CPY + ((c + bkt) & (CPY - 1))];
    if (t != 0) atomicAdd(&a.dtable[(int64_t)head * a.n_buckets + bkt], (float)((double)t * unscale));
  }
}

__global__ __launch_bounds__(256) void zero_f32_kernel(float* p, int n) {
  for (int t = threadIdx.x; t < n; t += 256) p[t] = 0.0f;
}

template <int DS, int NB>
void launch_short_t(const BwdArgs& a, hipStream_t s) {
  const int nseq = a.H / a.hpb;
  const int lgp = a.Sq > 128 ? 0 : (a.Sq > 64 ? 1 : (a.Sq > 32 ? 2 : 3));   // 2^lgp sequences per workgroup
  const int ngroups = (nseq + (1 << lgp) - 1) >> lgp;
  int slots = kMaxGridShort / a.hpb;
  if (slots < 1) slots = 1;
  if (slots > ngroups) slots = ngroups;
  const dim3 grid((unsigned)(slots * a.hpb));
  // row-wise staging reads 16 bytes from 4-byte aligned offsets
  const bool rows4 = reinterpret_cast<uintptr_t>(a.spd) % 4 == 0 && a.ld_spd % 4 == 0 &&
                     a.spd_bstride % 4 == 0;
  if constexpr (DS <= 16) {
    if (a.Sq % 32 == 0) {     // no keys past N in any block
      if (a.spd_t)
        hipLaunchKernelGGL((bwd_short_bf16_kernel<DS, NB, true, false, true>), grid, dim3(kThreads), 0, s, a);
      else if (rows4)
        hipLaunchKernelGGL((bwd_short_bf16_kernel<DS, NB, false, true, true>), grid, dim3(kThreads), 0, s, a);
      else
        hipLaunchKernelGGL((bwd_short_bf16_kernel<DS, NB, false, false, true>), grid, dim3(kThreads), 0, s, a);
      return;
    }
  }
  if (a.spd_t)
    hipLaunchKernelGGL((bwd_short_bf16_kernel<DS, NB, true, false>), grid, dim3(kThreads), 0, s, a);
  else if (rows4)
    hipLaunchKernelGGL((bwd_short_bf16_kernel<DS, NB, false, true>), grid, dim3(kThreads), 0, s, a);
  else
    hipLaunchKernelGGL((bwd_short_bf16_kernel<DS, NB, false, false>), grid, dim3(kThreads), 0, s, a);
}

template <int NB>
void launch_short_nb(const BwdArgs& a, int d, hipStream_t s) {
  switch (d) {
    case 8: launch_short_t<8, NB>(a, s); break;
    case 16: launch_short_t<16, NB>(a, s); break;
    default: launch_short_t<32, NB>(a, s); break;
  }
}

}  // namespace

bool bwd_short_applies(const BwdArgs& a, int d) {
  // (a group of up to 8 sequences is read through one resource of at most
  // 2^30 bytes)
  return d <= 32 && !a.accumulate && a.row_off == 0 && a.col_off == 0 && a.Sq == a.Sk &&
         a.Sq >= 1 && a.Sq <= kRows && a.hpb >= 1 && a.H % a.hpb == 0 &&
         (int64_t)8 * a.hpb * a.Sq * d * 2 < ((int64_t)1 << 30);
}

hipError_t launch_bwd_short_bf16(const BwdArgs& a, int d, hipStream_t s) {
  // dtable is cleared by a fill kernel (the workgroups add into it at their end)
  hipLaunchKernelGGL(zero_f32_kernel, dim3(1), dim3(256), 0, s, a.dtable, a.hpb * a.n_buckets);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (a.n_buckets <= 127)
    launch_short_nb<128>(a, d, s);
  else
    launch_short_nb<256>(a, d, s);
  return hipGetLastError();
}

}  // namespace gt
