// Backward, key-stationary stage: dK, dV and the bias-table gradient (bf16).
//
// Each wave owns 32 keys (lane & 31 = key) and streams every query through
// S = Q K^T with the queries on the MFMA rows, so the lane's registers hold
// P and dS for its key and 16 consecutive queries (lane half g: queries
// 16 g + r). Those registers are directly the B operands of
//   dV^T += dO^T P   and   dK^T += Q^T dS,
// with dO^T and Q^T read from LDS. The softmax statistics enter through the
// matrix-core accumulators: S starts from -LSE log2(e) / (scale log2(e)) and
// dP from -Dlt, so per score element the vector work is one FMA with the
// bias, one exp2, one multiply and the two bf16 conversions.
//
// Bias and table gradient: the table (times log2 e) is replicated in LDS
// (copy = lane & 31 when there are at most 128 buckets, else lane & 15) and
// the bucket histogram has the same layout, so
// one address register serves the bias read and the gradient add. The
// histogram is fixed point: LDS float atomics are slow on this hardware,
// 64-bit integer adds are not. dS is accumulated as round(dS * 2^F), where
// the power-of-two scale per head keeps every term below 2^30 in magnitude:
// |dS_ij| <= |dO_i . V_j - Dlt_i| <= max_i |dO_i| max_j |V_j| + max_i |Dlt_i|
// (P_ij <= 1, Cauchy-Schwarz), and the prepare stage records block maxima of
// |dO_i|, |V_j| and |Dlt_i|. Dlt enters on its own because in a ring step O
// mixes the values of every key block, not only of the keys at hand. The scale enters for free through the
// V operand of dP (and the dP accumulator start), so dS arrives already
// scaled; dK takes 2^-F in its final multiply. Sums of up to 2^32 terms fit
// in 64 bits. The histogram is flushed once per workgroup, converted back
// to fp32, with one global atomic per bucket.
//
// Query tiles (Q and dO row-major, statistics) are double buffered in LDS;
// Q^T and dO^T are read with transposing LDS reads. The next tile's global
// loads are in flight while the current one is computed, one barrier per
// tile. spd bytes are fetched one 32-query sub-block ahead of their use.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "stage.hpp"

namespace gt {

namespace {

constexpr int kNW = 8;              // waves per workgroup
constexpr int kBK = kNW * 32;       // keys per workgroup
constexpr int kBQ = 64;             // queries per staged tile
constexpr int kThreads = kNW * 64;
// Table / histogram copies: lane & (CPY - 1); 32 copies (two lanes per copy)
// in the 128-bucket layout, else 16.
template <int NB>
constexpr int copies() { return NB <= 128 ? 32 : 16; }

// All LDS of the kernel in one block, at LDS address 0: the staged tiles
// first (their offsets stay inside the reach of the DS immediate), then,
// from byte 64 KiB, the table copies and right after them the histogram
// copies. The per-element address register holds the absolute address of
// the table entry (bucket, copy); the histogram entry is at a fixed
// immediate offset (ENT * 8) from it. NB (128 or 256) bounds the byte
// values the layout covers.
template <int D>
struct DkdvTiles {
  uint16_t q[2][kBQ * D];
  uint16_t o[2][kBQ * D];
  float init_s[2][kBQ];             // -LSE log2 e / (scale log2 e); -inf for empty rows
  float init_p[2][kBQ];             // -Dlt 2^F
  float red[3][kNW];
  uint8_t stage[kNW][1024];         // per wave: a 32 x 32 block of spd bytes (row-wise staging)
};
constexpr uint32_t kTabBase = 65536;
template <int D, int NB>
struct DkdvSmem : DkdvTiles<D> {
  static constexpr int ENT = NB * copies<NB>();   // entry (b, c) = b * CPY + c
  uint8_t pad[kTabBase - sizeof(DkdvTiles<D>)];
  uint2 tabw[ENT];                  // table copies (fp32 bits, 8-byte stride)
  unsigned long long hist[ENT];     // gradient histogram copies, same index
};

// Per-lane LDS element offsets of the operand reads (tile-relative; the
// 32-query sub-block and 8-query step offsets are immediates).
template <int D>
struct DkdvOffsets {
  int row[D / 16];        // Q / dO rows perm32(lane), feature chunk 2 kc + g
  int tr[2][D / 32];      // transposing reads h = 0, 1, feature block cb
  __device__ __forceinline__ DkdvOffsets() {
#pragma unroll
    for (int kc = 0; kc < D / 16; ++kc) row[kc] = row_operand_off<D>(kc);
#pragma unroll
    for (int h = 0; h < 2; ++h)
#pragma unroll
      for (int cb = 0; cb < D / 32; ++cb) tr[h][cb] = tr_operand_off<D>(h, cb);
  }
};

// A query tile in flight: Q and dO rows (rows past N read as zero; source
// rows of DS < D features padded with zeros) and the statistics of its 64
// queries.
template <int D, int DS>
struct QTileStage {
  RowStage<D, kThreads, DS> q, o;
  float stat;

  __device__ __forceinline__ void load(const uint16_t* qh, const uint16_t* oh, const float* lse2h,
                                       const float* dlth, int64_t i0, int64_t n) {
    q.load(tile_rsrc<DS>(qh, i0, n));
    o.load(tile_rsrc<DS>(oh, i0, n));
    // every thread loads (two copies of the 128 values), clamped to row N-1
    const int ts = (int)threadIdx.x & (2 * kBQ - 1);
    const int64_t i = i0 + (ts & (kBQ - 1));
    const int64_t ic = i < n ? i : n - 1;
    stat = (ts < kBQ ? lse2h : dlth)[ic];
  }
  // Registers -> LDS buffer BUF, with the accumulator starts of S
  // (-lse2 / (scale log2 e), -inf for padded rows so that P = 0) and of the
  // scaled dP (-Dlt 2^F).
  template <int BUF, int NB>
  __device__ __forceinline__ void store(DkdvSmem<D, NB>& sm, int64_t i0, int64_t n, float inv_sl2,
                                        float sF) {
    q.store(sm.q[BUF]);
    o.store(sm.o[BUF]);
    const int t = threadIdx.x;
    if (t < 2 * kBQ) {
      float st = stat;
      opaque_f(st);
      const int qi = t & (kBQ - 1);
      const bool in = i0 + qi < n;
      if (t < kBQ)
        sm.init_s[BUF][qi] = in ? -st * inv_sl2 : -INFINITY;
      else
        sm.init_p[BUF][qi] = in ? -st * sF : 0.0f;
    }
  }
};

// spd bytes of this lane's key for the 16 queries i_base + 16 g + r, by raw
// buffer loads: a scalar base per sub-block, scalar row offsets r * ld and a
// per-lane offset 16 g ld + key. QFULL (N a multiple of the query tile): every
// row exists. Otherwise rows past n read the clamped row n-1 (their P is 0,
// any bucket will do), branch-free.
template <bool QFULL>
__device__ __forceinline__ void load_bytes(const uint8_t* spd_cols, int64_t ld, int64_t i_base,
                                           int64_t n, uint32_t key_off, uint8_t b[16]) {
  const int g = (threadIdx.x >> 5) & 1;
  if constexpr (QFULL) {
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(spd_cols + i_base * ld);
    const uint32_t voff = (uint32_t)(16 * g) * (uint32_t)ld + key_off;
#pragma unroll
    for (int r = 0; r < 16; ++r) b[r] = (uint8_t)buf_u8(rs, voff, (uint32_t)(r * ld));
  } else {
    // base at the clamped first row, so every offset below is >= 0
    const int64_t ib = i_base < n ? i_base : n - 1;
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(spd_cols + ib * ld);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      int64_t row = i_base + 16 * g + r;
      row = row < n ? row : n - 1;
      b[r] = (uint8_t)buf_u8(rs, (uint32_t)((row - ib) * ld) + key_off, 0u);
    }
  }
}

__device__ __forceinline__ int round_to_int(float x) {
  int r;
  asm("v_cvt_rpi_i32_f32 %0, %1" : "=v"(r) : "v"(x));   // floor(x + 0.5)
  return r;
}

// The 128-bucket layout is used only when n_buckets <= 127, so bucket 127
// is padding (bias 0, gradient discarded) and any byte of 128 or more, which
// has no entry in that layout, can be mapped to it. Valid inputs (buckets
// below n_buckets) never take the mapping branch.
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
template <int NB>
__device__ __forceinline__ void clamp_buckets(uint8_t (&b)[16]) {
  if constexpr (NB <= 128) {
    uint32_t any = 0;
#pragma unroll
    for (int r = 0; r < 16; ++r) any |= b[r];
    if (__any((any & 0x80u) != 0)) {
#pragma unroll
      for (int r = 0; r < 16; ++r) b[r] = (b[r] & 0x80u) ? (uint8_t)0x7f : b[r];
    }
  }
}

// b: this lane's 16 bucket indices, as 16 bytes (gathered from spd columns)
// or as 4 words (a 16-byte row segment of spd_t).
// STAGE: b holds 16 bytes of the block's spd rows (lane l: row l / 2 of the
// 32-query sub-block, bytes 16 (l % 2) .. + 15 of the wave's 32 keys); they
// are written to the wave's staging buffer and each lane reads its key's 16
// query bytes back with two 8-bit transposing reads (off_tr8).
template <int D, int NKS, int NB, bool KTAIL, int BUF, int QS, bool STAGE = false, typename BT>
__device__ __forceinline__ void dkdv_subblock(DkdvSmem<D, NB>& sm, const DkdvOffsets<D>& off,
                                              const bf16x8* kf, const bf16x8* vf,
                                              const BT* b, float sl2, bool jok,
                                              f32x16* dk, f32x16* dv, const int* off_tr8 = nullptr) {
  constexpr int NKC = D / 16;
  constexpr int NCB = D / 32;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 5;
  const int ib = QS * 32 + 16 * g;   // this lane half's first query in the tile

  f32x16 s, dp;
  {
    const float4* is4 = reinterpret_cast<const float4*>(&sm.init_s[BUF][ib]);
    const float4* ip4 = reinterpret_cast<const float4*>(&sm.init_p[BUF][ib]);
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const float4 x = is4[u], y = ip4[u];
      s[4 * u] = x.x; s[4 * u + 1] = x.y; s[4 * u + 2] = x.z; s[4 * u + 3] = x.w;
      dp[4 * u] = y.x; dp[4 * u + 1] = y.y; dp[4 * u + 2] = y.z; dp[4 * u + 3] = y.w;
    }
  }
#pragma unroll
  for (int kc = 0; kc < NKS; ++kc) {
    s = mfma32(lds_b128(sm.q[BUF] + QS * 32 * D + off.row[kc]), kf[kc], s);
    dp = mfma32(lds_b128(sm.o[BUF] + QS * 32 * D + off.row[kc]), vf[kc], dp);
  }
  // Lane: key; registers r: queries. dp holds (dO.V - Dlt) 2^F, so ds below
  // is dS 2^F.
  float p[16], ds[16];
  uint32_t addr[16];   // absolute LDS address of table entry (bucket, copy)
  float tb[16];
  constexpr int CPY = copies<NB>();
  // copy offset with the table base: kTabBase = 1 << 16 is byte 2, so a
  // byte permute can put the bucket into byte 1 and keep both
  const uint32_t cpyb = (uint32_t)(lane & (CPY - 1)) * 8u | kTabBase;
  if constexpr (sizeof(BT) == 4) {
    uint32_t w[4];
    if constexpr (STAGE) {
      typedef int i32x2 __attribute__((ext_vector_type(2)));
      typedef __attribute__((address_space(3))) i32x2* lds_i32x2;
      uint8_t* st8 = sm.stage[wave_id()];
      uint4 v4 = make_uint4(b[0], b[1], b[2], b[3]);
      opaque(v4);                                  // keep the load's wait here
      *reinterpret_cast<uint4*>(st8 + 16 * lane) = v4;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const i32x2 v = __builtin_amdgcn_ds_read_tr8_b64_v2i32((lds_i32x2)(void*)(st8 + off_tr8[hh]));
        w[2 * hh] = (uint32_t)v.x;
        w[2 * hh + 1] = (uint32_t)v.y;
      }
    } else {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        w[u] = b[u];
        opaque(w[u]);                              // keep the load's wait here
      }
    }
    clamp_buckets<NB>(w);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      if constexpr (CPY == 32)   // byte (r & 3) of w[r >> 2] times 256, plus copy and base
        addr[r] = __builtin_amdgcn_perm(w[r >> 2], cpyb, 0x0c020000u | ((4u + (r & 3)) << 8));
      else
        addr[r] = (((w[r >> 2] >> (8 * (r & 3))) & 0xffu) << 7) | cpyb;
    }
  } else {
    uint8_t bb[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      uint32_t bk = b[r];
      opaque(bk);                                  // keep the byte's wait here
      bb[r] = (uint8_t)bk;
    }
    clamp_buckets<NB>(bb);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const uint32_t bk = bb[r];
      if constexpr (CPY == 32)
        addr[r] = __builtin_amdgcn_perm(bk, cpyb, 0x0c020400u);   // byte0(bk) * 256 + copy + base
      else
        addr[r] = (bk << 7) | cpyb;
    }
  }
  const uint8_t* lds0 = reinterpret_cast<const uint8_t*>(&sm);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    tb[r] = *reinterpret_cast<const float*>(lds0 + addr[r]);
  }
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const float x = fmaf(s[r], sl2, tb[r]);
    float pv = exp2_fast(x);
    if constexpr (KTAIL) pv = jok ? pv : 0.0f;
    p[r] = pv;
    ds[r] = pv * dp[r];
  }
  constexpr uint32_t kHistOff = DkdvSmem<D, NB>::ENT * 8;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    unsigned long long* hp = reinterpret_cast<unsigned long long*>(const_cast<uint8_t*>(lds0) + addr[r] + kHistOff);
    const unsigned long long v = (unsigned long long)(long long)round_to_int(ds[r]);
    atomicAdd(hp, v);
  }
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const bf16x8 pb = cvt_bf16x8(p + 8 * q);
    const bf16x8 db = cvt_bf16x8(ds + 8 * q);
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
      const int base = (QS * 32 + 8 * q) * D;
      dv[cb] = mfma32(lds_tr_operand(sm.o[BUF] + base, off.tr[0][cb], off.tr[1][cb]), pb, dv[cb]);
      dk[cb] = mfma32(lds_tr_operand(sm.q[BUF] + base, off.tr[0][cb], off.tr[1][cb]), db, dk[cb]);
    }
  }
}

template <int D, int DS, int NB, bool KTAIL, bool QFULL, bool TR, bool STAGE>
__device__ __forceinline__ void dkdv_main(const BwdArgs& a, DkdvSmem<D, NB>& sm, int h, int64_t key0,
                                          int64_t j, bool jok, int fexp) {
  constexpr int NKC = D / 16;
  constexpr int NCB = D / 32;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 5;
  const int64_t hq = (int64_t)h * a.Sq * DS;   // query-side rows
  const int64_t hk = (int64_t)h * a.Sk * DS;   // key-side rows
  const uint16_t* qh = reinterpret_cast<const uint16_t*>(a.q) + hq;
  const uint16_t* kh = reinterpret_cast<const uint16_t*>(a.k) + hk;
  const uint16_t* vh = reinterpret_cast<const uint16_t*>(a.v) + hk;
  const uint16_t* oh = reinterpret_cast<const uint16_t*>(a.d_o) + hq;
  const float* lse2h = a.lse2 + (int64_t)h * a.Sq;
  const float* dlth = a.dlt + (int64_t)h * a.Sq;
  const float sl2 = a.scale * kLog2e;
  const float inv_sl2 = 1.0f / sl2;

  const float sF = ldexpf(1.0f, fexp);

  // K and 2^F V of this lane's key as B operands (rows past N: zero); the
  // power-of-two scale is exact in bf16.
  bf16x8 kf[NKC], vf[NKC];
#pragma unroll
  for (int kc = 0; kc < NKC; ++kc) {
    const bool in = jok && kc * 16 + g * 8 < DS;
    kf[kc] = in ? *reinterpret_cast<const bf16x8*>(kh + j * DS + kc * 16 + g * 8) : zero_bf16x8();
    const bf16x8 v8 = in ? *reinterpret_cast<const bf16x8*>(vh + j * DS + kc * 16 + g * 8) : zero_bf16x8();
#pragma unroll
    for (int e = 0; e < 8; ++e) vf[kc][e] = (__bf16)((float)v8[e] * sF);
  }
  f32x16 dk[NCB], dv[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    dk[cb] = zero_f32x16();
    dv[cb] = zero_f32x16();
  }

  const int64_t ld = a.ld_spd;
  const int64_t jc = jok ? j : a.Sk - 1;
  const uint32_t key_off = (uint32_t)(jc - key0);
  const uint8_t* spd_cols = seq_spd(a, h) + a.row_off * ld + a.col_off + key0;
  const int64_t ntiles = (a.Sq + kBQ - 1) / kBQ;
  const DkdvOffsets<D> off;

  // Bucket indices of this lane's key: TR reads 16 queries as one 16-byte
  // row segment of spd_t (rows of this key block only; past the block's last
  // row a load reads zeros), else gathers 16 bytes of a spd column.
  using BT = std::conditional_t<TR || STAGE, uint32_t, uint8_t>;
  constexpr int NBT = TR || STAGE ? 4 : 16;
  static_assert(!(TR && STAGE), "one way of reading spd");
  const __amdgpu_buffer_rsrc_t rs_t =
      make_rsrc_n(TR ? seq_spd_t(a, h) + key0 * ld : seq_spd(a, h), ((a.Sk - key0 < kBK ? a.Sk - key0 : kBK)) * ld);
  const uint32_t voff_t = (uint32_t)((jc - key0) * ld) + 16u * (uint32_t)g;
  // STAGE: lane l loads row l / 2 of the sub-block, bytes 16 (l % 2) .. + 15
  // of the wave's 32 keys, through a resource that starts at the sub-block's
  // first row and ends with the last query row (rows past Sq read zero); the
  // two transposing reads of the staged block give the lane its key's 16
  // query bytes.
  uint32_t voff_st = 0;
  int off_tr8[2] = {0, 0};
  if constexpr (STAGE) {
    voff_st = (uint32_t)((lane >> 1) * ld) + (uint32_t)(wave_id() * 32 + 16 * (lane & 1));
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
      off_tr8[hh] = (16 * g + 8 * hh + ((lane & 15) >> 1)) * 32 + 16 * ((lane >> 4) & 1) + 8 * (lane & 1);
  }
  auto fetch = [&](int64_t i_base, BT* dst) {
    if constexpr (TR) {
      buf_u128(rs_t, voff_t, (uint32_t)i_base, reinterpret_cast<uint32_t*>(dst));
    } else if constexpr (STAGE) {
      const int64_t ib = i_base < a.Sq ? i_base : a.Sq - 1;
      const __amdgpu_buffer_rsrc_t rs = make_rsrc_n(spd_cols + ib * ld, (a.Sq - ib) * ld);
      buf_u128(rs, voff_st + (uint32_t)((i_base - ib) * ld), 0u, reinterpret_cast<uint32_t*>(dst));
    } else {
      load_bytes<QFULL>(spd_cols, ld, i_base, a.Sq, key_off, reinterpret_cast<uint8_t*>(dst));
    }
  };

  QTileStage<D, DS> st;
  st.load(qh, oh, lse2h, dlth, 0, a.Sq);
  BT bA[NBT], bB[NBT];
  fetch(0, bA);
  st.template store<0>(sm, 0, a.Sq, inv_sl2, sF);
  wait_loads();
  __syncthreads();

  // One query tile on buffer BUF: the prefetches are unconditional (the last
  // tile re-reads itself), so every path has the same loads in flight and
  // the waits before each use stay exact.
  auto step = [&](int64_t t, auto bufc) {
    constexpr int BUF = decltype(bufc)::value;
    const int64_t i0 = t * kBQ;
    const bool more = t + 1 < ntiles;
    const int64_t inext = more ? i0 + kBQ : i0;
    fetch(i0 + 32, bB);
    st.load(qh, oh, lse2h, dlth, inext, a.Sq);
    sched_fence();
    dkdv_subblock<D, (DS + 15) / 16, NB, KTAIL, BUF, 0, STAGE>(sm, off, kf, vf, bA, sl2, jok, dk, dv, off_tr8);
    fetch(inext, bA);
    sched_fence();
    dkdv_subblock<D, (DS + 15) / 16, NB, KTAIL, BUF, 1, STAGE>(sm, off, kf, vf, bB, sl2, jok, dk, dv, off_tr8);
    if (more) st.template store<BUF ^ 1>(sm, inext, a.Sq, inv_sl2, sF);
    __syncthreads();
  };
  int64_t t = 0;
  for (; t + 1 < ntiles; t += 2) {
    step(t, std::integral_constant<int, 0>());
    step(t + 1, std::integral_constant<int, 1>());
  }
  if (t < ntiles) step(t, std::integral_constant<int, 0>());

  const float dk_scale = a.scale * ldexpf(1.0f, -fexp);
  if (jok && a.accumulate) {
    // fp32 partials of the key block, accumulated across ring steps
    float* dkp = reinterpret_cast<float*>(a.dk) + hk + j * DS;
    float* dvp = reinterpret_cast<float*>(a.dv) + hk + j * DS;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = cb * 32 + 8 * u + 4 * g;
        if (c >= DS) continue;               // zero padding of a narrow head dim
        float4 xk = *reinterpret_cast<const float4*>(dkp + c);
        float4 xv = *reinterpret_cast<const float4*>(dvp + c);
        xk.x += dk[cb][4 * u] * dk_scale; xk.y += dk[cb][4 * u + 1] * dk_scale;
        xk.z += dk[cb][4 * u + 2] * dk_scale; xk.w += dk[cb][4 * u + 3] * dk_scale;
        xv.x += dv[cb][4 * u]; xv.y += dv[cb][4 * u + 1];
        xv.z += dv[cb][4 * u + 2]; xv.w += dv[cb][4 * u + 3];
        *reinterpret_cast<float4*>(dkp + c) = xk;
        *reinterpret_cast<float4*>(dvp + c) = xv;
      }
    }
  } else if (jok) {
    uint16_t* dkp = reinterpret_cast<uint16_t*>(a.dk) + hk + j * DS;
    uint16_t* dvp = reinterpret_cast<uint16_t*>(a.dv) + hk + j * DS;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) {
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = cb * 32 + 8 * u + 4 * g;
        if (c >= DS) continue;
        uint2 pk, pv;
        pk.x = (uint32_t)f2bf(dk[cb][4 * u] * dk_scale) | ((uint32_t)f2bf(dk[cb][4 * u + 1] * dk_scale) << 16);
        pk.y = (uint32_t)f2bf(dk[cb][4 * u + 2] * dk_scale) | ((uint32_t)f2bf(dk[cb][4 * u + 3] * dk_scale) << 16);
        pv.x = (uint32_t)f2bf(dv[cb][4 * u]) | ((uint32_t)f2bf(dv[cb][4 * u + 1]) << 16);
        pv.y = (uint32_t)f2bf(dv[cb][4 * u + 2]) | ((uint32_t)f2bf(dv[cb][4 * u + 3]) << 16);
        *reinterpret_cast<uint2*>(dkp + c) = pk;
        *reinterpret_cast<uint2*>(dvp + c) = pv;
      }
    }
  }
}

// D: the tile's head dim (32 or 64); DS <= D: the head dim of the tensors
// (8 and 16 run on 32-wide tiles whose extra features are zero).
template <int D, int DS, int NB, bool QFULL, bool TR, bool STAGE = false>
__global__ __launch_bounds__(kThreads, 2) void bwd_dkdv_bf16_kernel(BwdArgs a) {
  constexpr int CPY = copies<NB>();
  __shared__ __attribute__((aligned(16))) DkdvSmem<D, NB> sm;
  uint2* tabw = sm.tabw;
  unsigned long long* hist = sm.hist;
  float (*red)[kNW] = sm.red;
  const int tid = threadIdx.x;
  const int wave = wave_id(), col = tid & 31;
  const int64_t nkb = (a.Sk + kBK - 1) / kBK;
  const int64_t lid = xcd_remap(blockIdx.x, nkb * a.H);
  const int h = (int)(lid % a.H);
  const int64_t kblk = lid / a.H;
  const int64_t j = kblk * kBK + wave * 32 + col;
  const bool jok = j < a.Sk;

  for (int t = tid; t < DkdvSmem<D, NB>::ENT; t += kThreads) {
    const int bkt = t / CPY;
    const float tv = (bkt < a.n_buckets) ? a.table[(int64_t)table_row(a, h) * a.n_buckets + bkt] * kLog2e : 0.0f;
    tabw[t] = make_uint2(__float_as_uint(tv), 0u);
    hist[t] = 0ull;
  }

  // Fixed-point exponent F of this head: (max|dO| max|V| + max|Dlt|) 2^F
  // <= 2^30 (a 1.5 % margin covers the rounding of P and of the products).
  {
    const int64_t nblk = ((a.Sq > a.Sk ? a.Sq : a.Sk) + 255) / 256;
    const float* nm = a.nmax + (int64_t)h * nblk * 4;
    float md = 0.0f, mv = 0.0f, ml = 0.0f;
    for (int64_t t = tid; t < nblk; t += kThreads) {
      md = fmaxf(md, nm[4 * t]);
      mv = fmaxf(mv, nm[4 * t + 1]);
      ml = fmaxf(ml, nm[4 * t + 2]);
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      md = fmaxf(md, __shfl_xor(md, off));
      mv = fmaxf(mv, __shfl_xor(mv, off));
      ml = fmaxf(ml, __shfl_xor(ml, off));
    }
    if ((tid & 63) == 0) {
      red[0][wave] = md;
      red[1][wave] = mv;
      red[2][wave] = ml;
    }
  }
  __syncthreads();
  float md = red[0][0], mv = red[1][0], ml = red[2][0];
#pragma unroll
  for (int w = 1; w < kNW; ++w) {
    md = fmaxf(md, red[0][w]);
    mv = fmaxf(mv, red[1][w]);
    ml = fmaxf(ml, red[2][w]);
  }
  const float bound = 1.015f * (sqrtf(md) * sqrtf(mv) + ml);
  int fexp = 40;
  if (bound > 0.0f && bound < INFINITY) {
    int e;
    frexpf(bound, &e);                 // bound < 2^e
    fexp = 30 - e;
    fexp = fexp > 40 ? 40 : (fexp < -100 ? -100 : fexp);
  }

  if ((kblk + 1) * kBK <= a.Sk)
    dkdv_main<D, DS, NB, false, QFULL, TR, STAGE>(a, sm, h, kblk * kBK, j, jok, fexp);
  else
    dkdv_main<D, DS, NB, true, QFULL, TR, STAGE>(a, sm, h, kblk * kBK, j, jok, fexp);

  __syncthreads();
  const double unscale = ldexp(1.0, -fexp);
  for (int bkt = tid; bkt < a.n_buckets; bkt += kThreads) {
    long long t = 0;
#pragma unroll
    for (int c = 0; c < CPY; ++c) t += (long long)hist[bkt * CPY + ((c + bkt) & (CPY - 1))];
    if (t != 0) atomicAdd(&a.dtable[(int64_t)table_row(a, h) * a.n_buckets + bkt], (float)((double)t * unscale));
  }
}

template <int D, int DS, int NB>
void launch_dkdv_t(const BwdArgs& a, hipStream_t s) {
  const int64_t nkb = (a.Sk + kBK - 1) / kBK;
  const dim3 grid((unsigned)(nkb * a.H));
  const bool qfull = a.Sq % kBQ == 0;
  if (a.spd_t) {
    if (qfull)
      hipLaunchKernelGGL((bwd_dkdv_bf16_kernel<D, DS, NB, true, true>), grid, dim3(kThreads), 0, s, a);
    else
      hipLaunchKernelGGL((bwd_dkdv_bf16_kernel<D, DS, NB, false, true>), grid, dim3(kThreads), 0, s, a);
  } else if (a.spd_vec) {
    // rows 16-byte aligned: row-wise loads staged through LDS
    hipLaunchKernelGGL((bwd_dkdv_bf16_kernel<D, DS, NB, true, false, true>), grid, dim3(kThreads), 0, s, a);
  } else {
    if (qfull)
      hipLaunchKernelGGL((bwd_dkdv_bf16_kernel<D, DS, NB, true, false>), grid, dim3(kThreads), 0, s, a);
    else
      hipLaunchKernelGGL((bwd_dkdv_bf16_kernel<D, DS, NB, false, false>), grid, dim3(kThreads), 0, s, a);
  }
}

template <int NB>
void launch_dkdv_nb(const BwdArgs& a, int d, hipStream_t s) {
  switch (d) {
    case 8: launch_dkdv_t<32, 8, NB>(a, s); break;
    case 16: launch_dkdv_t<32, 16, NB>(a, s); break;
    case 32: launch_dkdv_t<32, 32, NB>(a, s); break;
    default: launch_dkdv_t<64, 64, NB>(a, s); break;
  }
}

}  // namespace

hipError_t launch_dkdv_bf16(const BwdArgs& a, int d, hipStream_t s) {
  // Byte values at or past n_buckets read bias 0 and their gradient is
  // dropped. Up to 127 buckets the 128-bucket layout (one byte permute per
  // address) is used, with larger bytes mapped to its padding bucket 127;
  // otherwise the full 256-bucket layout.
  if (a.n_buckets <= 127)
    launch_dkdv_nb<128>(a, d, s);
  else
    launch_dkdv_nb<256>(a, d, s);
  return hipGetLastError();
}

}  // namespace gt
