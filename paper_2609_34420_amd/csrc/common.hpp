// Device-side building blocks shared by the gfx950 attention kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gt {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.69314718055994531f;

// 32x32x16 bf16 matrix-core product, fp32 accumulate (gfx950).
//   A operand: lane l supplies row (l & 31), k = (l >> 5) * 8 + [0, 8)
//   B operand: lane l supplies col (l & 31), k = (l >> 5) * 8 + [0, 8)
//   C/D:       lane l holds col (l & 31), rows 8u + 4 (l >> 5) + t in
//              register 4u + t (u, t in [0, 4))
__device__ __forceinline__ f32x16 mfma32(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// Index of the calling wave in its workgroup, as a wave-uniform (scalar)
// value: derived values such as buffer descriptors then stay in SGPRs.
__device__ __forceinline__ int wave_id() {
  return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
}

// Keep the compiler from moving instructions across this point (used after
// issuing prefetch loads, so no use of their results is hoisted next to
// them and forces an early wait).
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }

// Hide a loaded value from the optimiser until this point: nothing derived
// from it (e.g. the shifts that pack a transposed tile) can be computed
// earlier, next to the load, where it would force an early wait.
__device__ __forceinline__ void opaque(uint4& x) {
  asm volatile("" : "+v"(x.x), "+v"(x.y), "+v"(x.z), "+v"(x.w));
}
__device__ __forceinline__ void opaque(uint32_t& x) { asm volatile("" : "+v"(x)); }
__device__ __forceinline__ void opaque_f(float& x) { asm volatile("" : "+v"(x)); }

// Workgroup barrier that orders LDS accesses only: each wave waits for its
// own LDS operations (lgkmcnt), not for its global loads, so prefetches stay
// in flight across it. For kernels whose waves share nothing but LDS.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Wait for every outstanding vector-memory load (s_waitcnt vmcnt(0) with the
// other counters left free). Used once before a software-pipelined loop, so
// that values loaded ahead of it are not treated as pending inside the loop,
// where a conservative merge of the two loop entries would otherwise make the
// first use of the current tile also wait for the next tile's prefetch.
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// 2^x on the transcendental unit (v_exp_f32): exp2(-inf) = 0.
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

// Operand row permutation inside a 32-row block. If the A operand of a
// product loads block row perm32(m) into MFMA row m, then the C layout gives
// lane half g (lane >> 5) the 16 CONSECUTIVE block rows 16 g + r in its
// registers r = 0..15: C row 8u + 4g + t  <->  block row 16g + 4u + t.
// Consecutive rows per lane let one 16-byte load fetch the lane's spd bytes
// and let 8 consecutive registers feed the next product's operand.
__device__ __forceinline__ int perm32(int m) {
  return (((m >> 2) & 1) << 4) | ((m >> 3) << 2) | (m & 3);
}

__device__ __forceinline__ bf16x8 lds_b128(const uint16_t* p) {
  return *reinterpret_cast<const bf16x8*>(p);
}

__device__ __forceinline__ bf16x8 zero_bf16x8() {
  bf16x8 z;
#pragma unroll
  for (int i = 0; i < 8; ++i) z[i] = (__bf16)0.0f;
  return z;
}

__device__ __forceinline__ f32x16 zero_f32x16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.0f;
  return z;
}

__device__ __forceinline__ bf16x8 cvt_bf16x8(const float* x) {
  bf16x8 r;
#pragma unroll
  for (int i = 0; i < 8; ++i) r[i] = (__bf16)x[i];
  return r;
}

// Sum of the 8 bf16 values of v plus acc, by packed dot products with 1.
__device__ __forceinline__ float sum_bf16x8(const bf16x8& v, float acc) {
  const bf16x2 one = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
  for (int i = 0; i < 8; i += 2) {
    const bf16x2 pr = {v[i], v[i + 1]};
    acc = __builtin_amdgcn_fdot2_f32_bf16(pr, one, acc, false);
  }
  return acc;
}

// Weights of a pairwise LSE merge (Section III-A-1 part 3): a running state
// with log-sum-exp lo and a new block with lb combine to
// O = wo O_running + wb O_block, LSE = out. Two -inf inputs give weights 0 and
// out = -inf.
__device__ __forceinline__ void lse_merge_weights(float lo, float lb, float& wo, float& wb, float& out) {
  const float mx = fmaxf(lo, lb);
  if (mx == -INFINITY) {
    wo = 0.0f;
    wb = 0.0f;
    out = -INFINITY;
    return;
  }
  const float eo = expf(lo - mx), eb = expf(lb - mx);
  const float tot = eo + eb;
  wo = eo / tot;
  wb = eb / tot;
  out = mx + logf(tot);
}

__device__ __forceinline__ uint16_t f2bf(float x) {
  __bf16 b = (__bf16)x;
  return __builtin_bit_cast(uint16_t, b);
}

__device__ __forceinline__ float bf2f(uint16_t x) {
  return __uint_as_float(((uint32_t)x) << 16);
}

// Workgroup id -> logical id so that consecutive logical ids (the H heads of
// one row block, which share their spd tiles) land on the same XCD at about
// the same time. Workgroups are handed to the 8 XCDs round robin.
__device__ __forceinline__ int64_t xcd_remap(int64_t w, int64_t total) {
  if ((total & 7) != 0) return w;
  return (w & 7) * (total >> 3) + (w >> 3);
}

// Raw buffer resource over [base, base + 2 GiB): untyped loads, 32-bit data
// format (the gfx9-family descriptor word). Offsets passed to the loads below
// are always inside the caller's buffer; the range field is not relied on.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0x7fffffff, 0x00020000);
}

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t buf_u8(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff) {
  return (uint32_t)__builtin_amdgcn_raw_buffer_load_b8(r, voff, soff, 0);
}

__device__ __forceinline__ void buf_u128(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff,
                                         uint32_t w[4]) {
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
  w[0] = v[0]; w[1] = v[1]; w[2] = v[2]; w[3] = v[3];
}

// 16 spd bytes row[j .. j+15] as four dwords, byte by byte, bytes at or past
// `limit` read as 0. Used for unaligned slices and the last partial group;
// kept rolled so it costs few registers.
__device__ __forceinline__ void load_spd16_bytes(const uint8_t* row, int64_t j, int64_t limit,
                                                 uint32_t w[4]) {
  uint64_t lo = 0, hi = 0;
  const int64_t n = limit - j < 16 ? limit - j : 16;
#pragma unroll 1
  for (int t = 0; t < (int)n; ++t) {
    const uint64_t b = row[j + t];
    if (t < 8)
      lo |= b << (8 * t);
    else
      hi |= b << (8 * (t - 8));
  }
  w[0] = (uint32_t)lo; w[1] = (uint32_t)(lo >> 32);
  w[2] = (uint32_t)hi; w[3] = (uint32_t)(hi >> 32);
}


// spd bytes j .. j + KB - 1 (KB = 16 or 8) of a row into w (bytes past
// `limit` as 0, words past the block 0): one aligned load of KB bytes when
// `vec` (the whole block in range and the row 16-byte aligned), else bytes.
template <int KB>
__device__ __forceinline__ void load_spd_block(const uint8_t* row, int64_t j, int64_t limit, bool vec,
                                               uint32_t w[4]) {
  static_assert(KB == 16 || KB == 8, "spd block of 8 or 16 bytes");
  if (vec) {
    if constexpr (KB == 16) {
      const uint4 v4 = *reinterpret_cast<const uint4*>(row + j);
      w[0] = v4.x; w[1] = v4.y; w[2] = v4.z; w[3] = v4.w;
    } else {
      const uint2 v2 = *reinterpret_cast<const uint2*>(row + j);
      w[0] = v2.x; w[1] = v2.y; w[2] = 0; w[3] = 0;
    }
  } else {
    load_spd16_bytes(row, j, limit - j < KB ? limit : j + KB, w);
  }
}

// LDS tiles of the fp32 vector-ALU kernels. Each of the 16 threads of a row
// reads its own block of GB consecutive tile rows, so at any one read the
// threads are GB rows apart. Tile row r is kept at LDS row r + r / GB with a
// row stride of D + 4 floats: thread s then reads LDS row s (GB + 1) + k,
// and for D = 8, 16, 32, 64 the 16 threads' 16-byte reads fall in distinct
// bank groups. Without the padding and the gap they would all hit the same
// banks.
template <int D>
constexpr int valu_row_stride() { return D + 4; }
template <int R, int GB>
constexpr int valu_tile_rows() { return R + R / GB; }
template <int GB>
__device__ __forceinline__ int valu_row(int r) { return r + r / GB; }

// Rows r0 .. r0 + R - 1 of two row-major fp32 [nrows, D] tensors into LDS
// tiles (the layout above) by NT threads, rows past nrows as zero, in
// 16-byte loads and stores. x and y are 16-byte aligned: the entry points
// reject unaligned tensors, and a head's rows start at a multiple of 16
// bytes since D is a multiple of 4.
template <int R, int D, int GB, int NT>
__device__ __forceinline__ void stage_rows_f32(const float* x, const float* y, int64_t r0, int64_t nrows,
                                               float (*sx)[valu_row_stride<D>()],
                                               float (*sy)[valu_row_stride<D>()]) {
  static_assert(D % 4 == 0, "rows of whole 16-byte chunks");
  for (int t = (int)threadIdx.x; t < R * D / 4; t += NT) {
    const int r = t / (D / 4), c = (t % (D / 4)) * 4;
    float4 u = make_float4(0.0f, 0.0f, 0.0f, 0.0f), v = u;
    if (r0 + r < nrows) {
      u = *reinterpret_cast<const float4*>(x + (r0 + r) * D + c);
      v = *reinterpret_cast<const float4*>(y + (r0 + r) * D + c);
    }
    *reinterpret_cast<float4*>(&sx[valu_row<GB>(r)][c]) = u;
    *reinterpret_cast<float4*>(&sy[valu_row<GB>(r)][c]) = v;
  }
}

// The same tiles through registers: load() issues the 16-byte loads of a
// tile, store() writes them to LDS, so the loads of the next tile are in
// flight while the current one is computed (2 R D / NT floats per thread).
template <int R, int D, int GB, int NT>
struct RowPrefetchF32 {
  static_assert(D % 4 == 0 && (R * D / 4) % NT == 0, "whole 16-byte chunks, evenly over the threads");
  static constexpr int N = R * D / 4 / NT;
  float4 u[N], v[N];
  __device__ __forceinline__ void load(const float* x, const float* y, int64_t r0, int64_t nrows) {
#pragma unroll
    for (int s = 0; s < N; ++s) {
      const int t = (int)threadIdx.x + s * NT;
      const int r = t / (D / 4), c = (t % (D / 4)) * 4;
      u[s] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      v[s] = u[s];
      if (r0 + r < nrows) {
        u[s] = *reinterpret_cast<const float4*>(x + (r0 + r) * D + c);
        v[s] = *reinterpret_cast<const float4*>(y + (r0 + r) * D + c);
      }
    }
  }
  __device__ __forceinline__ void store(float (*sx)[valu_row_stride<D>()], float (*sy)[valu_row_stride<D>()]) const {
#pragma unroll
    for (int s = 0; s < N; ++s) {
      const int t = (int)threadIdx.x + s * NT;
      const int r = t / (D / 4), c = (t % (D / 4)) * 4;
      *reinterpret_cast<float4*>(&sx[valu_row<GB>(r)][c]) = u[s];
      *reinterpret_cast<float4*>(&sy[valu_row<GB>(r)][c]) = v[s];
    }
  }
};

// Row `row` of a row-major fp32 [*, D] tensor (16-byte aligned rows) times
// `mul` into registers, or zeros when !ok. The row is read unconditionally
// (callers pass a valid row, clamped when !ok) in 16-byte loads that are
// all in flight together, rather than one guarded load and wait per element.
template <int D>
__device__ __forceinline__ void load_row_f32(const float* base, int64_t row, bool ok, float mul, float (&out)[D]) {
  const float4* p = reinterpret_cast<const float4*>(base + row * D);
  const float f = ok ? mul : 0.0f;
#pragma unroll
  for (int c = 0; c < D / 4; ++c) {
    const float4 x = p[c];
    out[4 * c] = x.x * f;
    out[4 * c + 1] = x.y * f;
    out[4 * c + 2] = x.z * f;
    out[4 * c + 3] = x.w * f;
  }
}
}  // namespace gt
