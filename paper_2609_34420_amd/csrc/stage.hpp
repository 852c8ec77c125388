// Row-major LDS tiles of 64 rows x D bf16, staged global -> registers ->
// LDS, and the two ways the products read them:
//   * as an operand whose contraction runs along the row (K in S = Q K^T):
//     one 16-byte read per lane;
//   * as an operand whose contraction runs DOWN the rows (V in O = P V, K in
//     dQ = dS K, Q and dO in dK = dS^T Q, dV = P^T dO): two transposing
//     8-byte reads (ds_read_b64_tr_b16) per lane, so no tile is ever stored
//     transposed and no register shuffling is needed.
//
// Transposing read, per 16-lane group: lane L receives element (L & 3) of the
// 8 bytes read by lane 4 e + (L >> 2), for e = 0..3. If lane s of the group
// reads row R + (s >> 2), columns C + 4 (s & 3) .. + 3, lane L therefore
// receives column C + L of rows R .. R + 3: a 4 x 16 block arrives
// transposed.
#pragma once
#include "common.hpp"

namespace gt {

constexpr int kTileRows = 64;

// XOR swizzle of the 16-byte chunks of a tile row. Chosen (by exhaustive
// search over XORs of up to two row bits per chunk bit) so that the tile
// store (8 lanes per row), the row-operand reads (rows perm32(lane)) and the
// transposing reads (4 rows x 4 column groups per 16 lanes) are all free of
// bank conflicts, for a 64-bank LDS in 16-lane groups and a 32-bank LDS in
// 8-lane groups. Row bits 3 and 5 are not used, so rows 8 and 32 apart share
// one per-lane address pattern (their offsets are immediates).
template <int D>
__device__ __forceinline__ int swz_tile(int row, int chunk) {
  if constexpr (D == 64)
    return chunk ^ (((row >> 1) & 1) | (((row ^ (row >> 2)) & 1) << 1) |
                    ((((row >> 1) ^ (row >> 4)) & 1) << 2));
  else
    return chunk ^ (((row >> 4) & 1) | ((((row >> 1) ^ (row >> 2)) & 1) << 1));
}

// Raw buffer resource over exactly nbytes: loads past the end return 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc_n(const void* base, int64_t nbytes) {
  const int n = (int)(nbytes < 0x7fffffff ? nbytes : 0x7fffffff);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, n, 0x00020000);
}

// Resource over rows [r0, min(r0 + 64, nrows)) of a row-major [nrows, D]
// bf16 tensor: the tile's rows past nrows read as zero.
template <int D>
__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const uint16_t* t, int64_t r0, int64_t nrows) {
  const int64_t rows = nrows - r0 < kTileRows ? nrows - r0 : kTileRows;
  return make_rsrc_n(t + r0 * D, rows * D * 2);
}

__device__ __forceinline__ uint4 buf_b128(__amdgpu_buffer_rsrc_t r, uint32_t voff) {
  const u32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, 0, 0);
  return make_uint4(v[0], v[1], v[2], v[3]);
}

// Source rows narrower than the tile (DS < D features, for head dims 8 and
// 16 on the 32-wide tiles): a chunk at or past DS / 8 is loaded from this
// offset, past the end of every tile resource, so the load returns zeros.
constexpr uint32_t kZeroChunk = 0x40000000u;

// Byte offset, in a tile of DS-feature source rows, of 16-byte chunk `chunk`
// of row `row` (zero-filled past DS).
template <int DS>
__device__ __forceinline__ uint32_t src_chunk_off(int row, int chunk) {
  return chunk < DS / 8 ? (uint32_t)(row * DS * 2 + chunk * 16) : kZeroChunk;
}

// One tensor's tile in flight: NT threads, 16 bytes per item, item u =
// row u / (D/8), chunk u % (D/8); the source rows hold DS <= D features (a
// tile of them is contiguous in global memory) and the chunks past DS read
// as zero. With fewer items than threads, the extra threads load a
// duplicate (so every wave issues the same loads) and store nothing.
template <int D, int NT, int DS = D>
struct RowStage {
  static constexpr int CPR = D / 8;
  static constexpr int ITEMS = kTileRows * CPR;
  static constexpr int IPT = ITEMS >= NT ? ITEMS / NT : 1;
  static_assert(ITEMS % NT == 0 || NT % ITEMS == 0, "tile items must divide evenly");
  uint4 r[IPT];

  __device__ __forceinline__ static int item(int s) {
    return ITEMS >= NT ? (int)threadIdx.x + s * NT : (int)threadIdx.x % ITEMS;
  }
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs) {
#pragma unroll
    for (int s = 0; s < IPT; ++s) {
      if constexpr (DS == D)
        r[s] = buf_b128(rs, (uint32_t)item(s) * 16u);
      else
        r[s] = buf_b128(rs, src_chunk_off<DS>(item(s) / CPR, item(s) % CPR));
    }
  }
  // LDS element offset of this thread's item s.
  __device__ __forceinline__ static int lds_off(int s) {
    const int u = item(s);
    const int row = u / CPR;
    return row * D + swz_tile<D>(row, u % CPR) * 8;
  }
  __device__ __forceinline__ void store(uint16_t* tile) {
    if (ITEMS >= NT || (int)threadIdx.x < ITEMS) {
#pragma unroll
      for (int s = 0; s < IPT; ++s) {
        uint4 v = r[s];
        opaque(v);
        *reinterpret_cast<uint4*>(tile + lds_off(s)) = v;
      }
    }
  }
};

// Direct global -> LDS copy (buffer_load_dwordx4 ... lds): each lane's 16
// bytes land at the wave-uniform LDS base + 16 lane, and lanes past the
// descriptor's range write zeros. A pair of tiles (64 rows x D bf16 each,
// one descriptor per tensor) is split into 1 KiB blocks handed to the NW
// waves in order; within a block, lane l fills LDS chunk l % (D/8) of tile
// row (block row 0) + l / (D/8), so it reads the logical chunk that the
// swizzle stores there. Source rows of DS < D features leave the chunks
// past DS zero.
template <int D, int NW, int DS = D>
struct TileDma {
  static constexpr int ROWB = D * 2;
  static constexpr int RPB = 1024 / ROWB;              // rows per block
  static constexpr int NBLK = kTileRows * ROWB / 1024; // blocks per tensor
  static constexpr int BPW = 2 * NBLK / NW;            // blocks per wave
  static_assert(2 * NBLK % NW == 0, "blocks must divide evenly over the waves");
  static constexpr int NLOADS = BPW;                   // vector-memory ops per wave per tile pair
  uint32_t voff[BPW];
  int second[BPW], lds_byte[BPW];                      // wave-uniform

  __device__ __forceinline__ explicit TileDma(int wave) {
    const int lane = threadIdx.x & 63;
#pragma unroll
    for (int i = 0; i < BPW; ++i) {
      const int gb = wave * BPW + i;
      const int lb = gb % NBLK;
      second[i] = gb / NBLK;
      lds_byte[i] = lb * 1024;
      const int row = lb * RPB + lane / (D / 8);
      const int chunk = swz_tile<D>(row, lane % (D / 8));   // involution: logical chunk here
      if constexpr (DS == D)
        voff[i] = (uint32_t)(row * ROWB + chunk * 16);
      else
        voff[i] = src_chunk_off<DS>(row, chunk);
    }
  }
  __device__ __forceinline__ void load(__amdgpu_buffer_rsrc_t rs0, __amdgpu_buffer_rsrc_t rs1,
                                       uint16_t* dst0, uint16_t* dst1) const {
    typedef __attribute__((address_space(3))) void* lds_void;
#pragma unroll
    for (int i = 0; i < BPW; ++i) {
      uint8_t* base = reinterpret_cast<uint8_t*>(second[i] ? dst1 : dst0) + lds_byte[i];
      // Device pass only: in the host pass of this source the builtin stops
      // the host-side launch stubs of the kernels that use it from being emitted.
#if __HIP_DEVICE_COMPILE__
      __builtin_amdgcn_raw_ptr_buffer_load_lds(second[i] ? rs1 : rs0, (lds_void)(void*)base, 16, voff[i], 0, 0, 0);
#else
      (void)base;
      (void)rs0;
      (void)rs1;
#endif
    }
  }
};

// s_waitcnt vmcnt(N), other counters free.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Per-lane element offset of the row-operand read of rows perm32(lane & 31)
// (+ 32 sb as an immediate), feature chunk 2 kc + (lane >> 5).
template <int D>
__device__ __forceinline__ int row_operand_off(int kc) {
  const int lane = threadIdx.x & 63;
  const int row = perm32(lane & 31);
  return row * D + swz_tile<D>(row, 2 * kc + (lane >> 5)) * 8;
}

// Per-lane element offset of transposing read h (0, 1) for output rows
// (features) 32 cb .. 32 cb + 31: the lane half g covers tile rows
// 16 g + 4 h .. + 3 (+ 8 q + 32 sb as immediates).
template <int D>
__device__ __forceinline__ int tr_operand_off(int h, int cb) {
  const int lane = threadIdx.x & 63;
  const int s = lane & 15;
  const int row = 16 * (lane >> 5) + 4 * h + (s >> 2);
  const int col = 32 * cb + 16 * ((lane >> 4) & 1) + 4 * (s & 3);
  return row * D + swz_tile<D>(row, col >> 3) * 8 + (col & 4);
}

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));

__device__ __forceinline__ s16x4 lds_tr16(const uint16_t* p) {
  typedef __attribute__((address_space(3))) s16x4* lds_ptr;
  return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_ptr)(uint16_t*)p);
}

// A-operand of a 32x32x16 product whose rows are tile COLUMNS 32 cb + (lane
// & 31) and whose k index 8 g + j (g = lane >> 5) is tile row base + 16 g + j
// (base = 8 q + 32 sb): the transposed view of the tile, two reads.
__device__ __forceinline__ bf16x8 lds_tr_operand(const uint16_t* tile, int off0, int off1) {
  const s16x4 a = lds_tr16(tile + off0);
  const s16x4 b = lds_tr16(tile + off1);
  const s16x8 c = __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, c);
}


// Per-lane bias table in LDS for the query-stationary kernels: every byte
// value 0..255 has an entry (0 at or past n_buckets), one copy per lane,
// entry (b, lane) at byte 256 b + 4 lane, holding table[h, b] / scale. A
// score accumulator started from these entries and advanced by the matrix
// cores holds bias / scale + q.k.
constexpr int kLaneTableFloats = 256 * 64;

__device__ __forceinline__ void fill_lane_table(float* tab, const float* table_h, int n_buckets,
                                                float scale, int nthreads) {
  const float inv_scale = 1.0f / scale;
  // 16 bytes (4 lanes' copies of one bucket) per store
  for (int t = (int)threadIdx.x; t < kLaneTableFloats / 4; t += nthreads) {
    const int b = t >> 4;
    const float x = (b < n_buckets) ? table_h[b] * inv_scale : 0.0f;
    reinterpret_cast<float4*>(tab)[t] = make_float4(x, x, x, x);
  }
}

// Bias entries of this lane's 16 keys (4 spd words) loaded into a score
// accumulator: entry address 256 b + 4 lane from one byte permute.
__device__ __forceinline__ void load_bias(const float* tab, const uint32_t (&w)[4], uint32_t lane4,
                                          f32x16& s) {
  const uint8_t* tb = reinterpret_cast<const uint8_t*>(tab);
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const uint32_t addr = __builtin_amdgcn_perm(w[r >> 2], lane4, 0x0c0c0000u | ((4u + (r & 3)) << 8));
    s[r] = *reinterpret_cast<const float*>(tb + addr);
  }
}

}  // namespace gt
