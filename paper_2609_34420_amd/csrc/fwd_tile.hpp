// Building blocks of the bf16 forward kernels (the full forward / ring step
// in fwd.hip and the persistent short-sequence forward in fwd_short.hip):
// the per-lane softmax state, the operand offsets, the score product with
// the bias as its accumulator start, and the softmax of one 32 x 32 block
// with its P^T V product (the lazy reference is described in fwd.hip).
#pragma once
#include "common.hpp"
#include "stage.hpp"

namespace gt {

namespace {

constexpr float kBlockSumLimit = 256.0f;

// Softmax state of one 32-query block (per lane: one query, one lane half).
struct SoftmaxState {
  float m;        // reference max (log2 units), -inf before any finite score
  float mneg;     // -m, or 0 while m = -inf
  float l;        // this lane half's partial row sum, relative to m
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


// p = 2^x for the lane's 16 keys, as two bf16x8 operands, and their sum.
__device__ __forceinline__ float exp_block(const float (&x)[16], bf16x8& p0, bf16x8& p1) {
  float p[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) p[r] = exp2_fast(x[r]);
  p0 = cvt_bf16x8(p);
  p1 = cvt_bf16x8(p + 8);
  return sum_bf16x8(p1, sum_bf16x8(p0, 0.0f));
}

// Softmax of one 32x32 score block s (accumulated as bias/scale + q.k) and
// its P^T V product into acc. The exact path runs only when some lane's
// block sum exceeds the limit (or is not finite) or a row has no reference.
template <int D, bool MASK>
__device__ __forceinline__ void softmax_pv(const f32x16& s, const bf16x8 (&vop)[2][D / 32],
                                           int64_t jrem, float sl2, SoftmaxState& st,
                                           f32x16 (&acc)[D / 32]) {
  constexpr int NCB = D / 32;
  const int g = (threadIdx.x >> 5) & 1;
  float x[16];
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const float xv = fmaf(s[r], sl2, st.mneg);
    if constexpr (MASK)
      x[r] = (16 * g + r < jrem) ? xv : -INFINITY;
    else
      x[r] = xv;
  }
  bf16x8 p0, p1;
  float bs = exp_block(x, p0, p1);
  if (__any(!(bs <= kBlockSumLimit) || st.m == -INFINITY)) {
    // Exact path: move the reference to the row max of this block. x holds
    // scores relative to the old reference (absolute while there is none).
    float mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) mx = fmaxf(mx, x[r]);
    mx -= st.mneg;
    const float mall = fmaxf(mx, __shfl_xor(mx, 32));
    const float mnew = fmaxf(st.m, mall);
    const float alpha = (mnew == -INFINITY) ? 1.0f : exp2_fast(st.m - mnew);
    st.l *= alpha;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[cb][r] *= alpha;
    const float mneg_new = (mnew == -INFINITY) ? 0.0f : -mnew;
    const float shift = mneg_new - st.mneg;
    st.m = mnew;
    st.mneg = mneg_new;
#pragma unroll
    for (int r = 0; r < 16; ++r) x[r] += shift;
    bs = exp_block(x, p0, p1);
  }
  st.l += bs;
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    acc[cb] = mfma32(vop[0][cb], p0, acc[cb]);
    acc[cb] = mfma32(vop[1][cb], p1, acc[cb]);
  }
}

// Score product of one 32x32 unit: bias entries into the accumulator, then
// the K operands of key block kb (read from the staged tile) times the
// unit's Q^T.
// NK: the 16-feature chunks that hold data (all D / 16, or fewer when the
// source rows are narrower than the tile and the rest is zero).
template <int D, int NK>
__device__ __forceinline__ void issue_scores(const float* tab, const uint32_t (&w)[4], uint32_t lane4,
                                             const uint16_t* sK, const int (&koff)[D / 16], int kb,
                                             const bf16x8 (&q)[D / 16], f32x16& s) {
  load_bias(tab, w, lane4, s);
#pragma unroll
  for (int kc = 0; kc < NK; ++kc) s = mfma32(lds_b128(sK + kb * 32 * D + koff[kc]), q[kc], s);
}

template <int D>
__device__ __forceinline__ void read_v(const uint16_t* sV, const FwdOffsets<D>& off, int kb,
                                       bf16x8 (&vop)[2][D / 32]) {
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int cb = 0; cb < D / 32; ++cb)
      vop[q][cb] = lds_tr_operand(sV + (kb * 32 + 8 * q) * D, off.v[0][cb], off.v[1][cb]);
}

}  // namespace

}  // namespace gt
