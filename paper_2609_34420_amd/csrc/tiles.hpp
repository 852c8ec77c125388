// Double-buffered staging of key/value tiles for the query-stationary
// kernels (forward, ring step, dQ): global -> registers for tile t+1 while
// tile t is computed, then registers -> LDS, one barrier per tile.
#pragma once
#include "common.hpp"

namespace gt {

// Tile of BC = 64 keys. Each work item is a pair of key rows x one 16-byte
// feature chunk, so a transposed copy can be written as packed dwords.
//   K_ROW : K row-major (A operand of S^T = K Q^T)
//   K_T   : K^T        (A operand of dQ^T = K^T dS^T)
//   V_ROW : V row-major (A operand of dP^T = V dO^T)
//   V_T   : V^T        (A operand of O^T = V^T P^T)
template <int D, int NT, bool K_ROW, bool K_T, bool V_ROW, bool V_T>
struct KVStager {
  static constexpr int BC = 64;
  static constexpr int CPR = D / 8;
  static constexpr int ITEMS = (BC / 2) * CPR;        // per tensor
  static constexpr int TOTAL = 2 * ITEMS;             // K items then V items
  static constexpr int IPT = (TOTAL + NT - 1) / NT;   // items per thread

  uint4 r0[IPT], r1[IPT];

  // Rows past nk are loaded from the clamped row nk-1 (always in bounds, so
  // the loads are unconditional and never wait on a masked-lane write) and
  // zeroed by mask_tail().
  __device__ __forceinline__ void load(const uint16_t* kh, const uint16_t* vh, int64_t j0, int64_t nk) {
#pragma unroll
    for (int s = 0; s < IPT; ++s) {
      const int it = (int)threadIdx.x + s * NT;
      if (TOTAL % NT == 0 || it < TOTAL) {
        const int u = it % ITEMS;
        const int jp = u % (BC / 2), cc = u / (BC / 2);
        const uint16_t* src = (it < ITEMS) ? kh : vh;
        const int64_t row = j0 + 2 * jp;
        const int64_t r0c = row < nk ? row : nk - 1;
        const int64_t r1c = row + 1 < nk ? row + 1 : nk - 1;
        r0[s] = *reinterpret_cast<const uint4*>(src + r0c * D + cc * 8);
        r1[s] = *reinterpret_cast<const uint4*>(src + r1c * D + cc * 8);
      }
    }
  }

  // Zero the rows of a partial last tile (a uniform branch around it).
  __device__ __forceinline__ void mask_tail(int64_t j0, int64_t nk) {
#pragma unroll
    for (int s = 0; s < IPT; ++s) {
      const int it = (int)threadIdx.x + s * NT;
      const int u = it % ITEMS;
      const int64_t row = j0 + 2 * (u % (BC / 2));
      if (row >= nk) r0[s] = make_uint4(0, 0, 0, 0);
      if (row + 1 >= nk) r1[s] = make_uint4(0, 0, 0, 0);
    }
  }

  __device__ __forceinline__ static void put_rows(uint16_t* dst, int row, int cc, const uint4& a, const uint4& b) {
    *reinterpret_cast<uint4*>(dst + row * D + swz_rows<D>(row, cc) * 8) = a;
    *reinterpret_cast<uint4*>(dst + (row + 1) * D + swz_rows<D>(row + 1, cc) * 8) = b;
  }

  __device__ __forceinline__ static void put_t(uint16_t* dst, int row, int cc, const uint4& a, const uint4& b) {
    const uint16_t* p0 = reinterpret_cast<const uint16_t*>(&a);
    const uint16_t* p1 = reinterpret_cast<const uint16_t*>(&b);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int crow = cc * 8 + e;
      *reinterpret_cast<uint32_t*>(dst + crow * BC + swz_t64(crow, row >> 3) * 8 + (row & 7)) =
          (uint32_t)p0[e] | ((uint32_t)p1[e] << 16);
    }
  }

  // k_row, k_t, v_row, v_t: LDS tiles of this buffer (unused ones may be null)
  __device__ __forceinline__ void store(uint16_t* k_row, uint16_t* k_t, uint16_t* v_row, uint16_t* v_t) {
#pragma unroll
    for (int s = 0; s < IPT; ++s) {
      const int it = (int)threadIdx.x + s * NT;
      if (TOTAL % NT == 0 || it < TOTAL) {
        const int u = it % ITEMS;
        const int jp = u % (BC / 2), cc = u / (BC / 2);
        const int row = 2 * jp;
        uint4 a = r0[s], b = r1[s];
        opaque(a);
        opaque(b);
        if (it < ITEMS) {
          if constexpr (K_ROW) put_rows(k_row, row, cc, a, b);
          if constexpr (K_T) put_t(k_t, row, cc, a, b);
        } else {
          if constexpr (V_ROW) put_rows(v_row, row, cc, a, b);
          if constexpr (V_T) put_t(v_t, row, cc, a, b);
        }
      }
    }
  }
};

}  // namespace gt
