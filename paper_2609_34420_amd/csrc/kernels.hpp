// Kernel argument blocks and host-side launchers (internal to libgtattn).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gt {

// Biased attention of a query block against a key block with the bias slice
// aligned by global offsets. Serves both the full forward (offsets 0,
// ld = N) and one context-parallel ring step.
struct FwdArgs {
  const void* q;          // [H, Sq, d]
  const void* k;          // [H, Sk, d]
  const void* v;          // [H, Sk, d]
  const uint8_t* spd;     // element (r, c) at spd[r * ld_spd + c]
  int64_t ld_spd;
  int64_t row_off;        // spd row of query 0
  int64_t col_off;        // spd column of key 0
  const float* table;     // [H, n_buckets]
  int32_t n_buckets;
  void* o;                // [H, Sq, d] (bf16 or fp32)
  float* lse;             // [H, Sq] natural log
  int32_t H;
  int64_t Sq;
  int64_t Sk;
  float scale;            // multiplies Q K^T
  int32_t spd_vec;        // every 16-byte spd group is 16-byte aligned
  int32_t accumulate;     // 1 (fp32 outputs only): o, lse hold a running merged state and
                          // this block is merged into it in place
  int32_t hpb;            // heads per sequence: "head" h of H is head h % hpb of sequence h / hpb
  int64_t spd_bstride;    // bytes from one sequence's spd to the next (0: one spd for all)
};

// Backward of a query block (Sq rows: q, o, d_o, lse, dq and the workspace
// rows) against a key block (Sk rows: k, v, dk, dv). The full backward has
// Sq = Sk = N and zero offsets; a context-parallel ring step has the rank's
// query shard, the KV block it holds and their global spd offsets.
struct BwdArgs {
  const void* q;
  const void* k;
  const void* v;
  const uint8_t* spd;     // (query i, key j) at spd[(row_off + i) * ld_spd + col_off + j]
  const uint8_t* spd_t;   // transpose of spd (same ld, zero offsets), or null: gather columns
  int64_t ld_spd;
  int64_t row_off;
  int64_t col_off;
  const float* table;
  int32_t n_buckets;
  const void* o;
  const float* lse;
  const void* d_o;
  void* dq;
  void* dk;
  void* dv;
  float* dtable;
  float* lse2;            // workspace [H, N]: LSE * log2(e), +inf for empty rows
  float* dlt;             // workspace [H, N]: rowsum(dO * O)
  float* nmax;            // workspace [H, ceil(max(Sq, Sk)/256), 4]: per block of 256 rows the
                          // max of |dO_i|^2, |V_j|^2, |Dlt_i| (and one pad)
  int32_t H;
  int64_t Sq;
  int64_t Sk;
  float scale;
  int32_t spd_vec;        // every 16-byte spd group of the block is 16-byte aligned
  int32_t accumulate;     // 1: dq, dk, dv are fp32 and receive +=; dtable is not cleared
  int32_t hpb;            // heads per sequence: "head" h of H is head h % hpb of sequence h / hpb
                          // (table and dtable rows are per head, shared by the sequences)
  int64_t spd_bstride;    // bytes from one sequence's spd (and spd_t) to the next (0: shared)
};

// A batch of sequences runs as H = B * hpb "heads": the table row of head h
// and the spd (spd_t) of its sequence.
template <typename Args>
__device__ __forceinline__ int table_row(const Args& a, int h) { return h % a.hpb; }
template <typename Args>
__device__ __forceinline__ const uint8_t* seq_spd(const Args& a, int h) {
  return a.spd + (int64_t)(h / a.hpb) * a.spd_bstride;
}
__device__ __forceinline__ const uint8_t* seq_spd_t(const BwdArgs& a, int h) {
  return a.spd_t + (int64_t)(h / a.hpb) * a.spd_bstride;
}

struct MergeArgs {
  const float* o_parts;   // [P, H, S, d]
  const float* lse_parts; // [P, H, S]
  int32_t n_parts;
  void* o;                // [H, S, d]
  float* lse;             // [H, S]
  int64_t rows;           // H * S
  int32_t d;
};

// Launchers return the hipError_t of the launch.
hipError_t launch_fwd(const FwdArgs& a, int d, bool bf16, bool out_f32, hipStream_t s);
// Sequences of at most 256 rows, N a multiple of 4 (bf16 in and out,
// d <= 32, at most 127 buckets, spd rows 4-byte aligned): the persistent
// whole-sequence forward.
bool fwd_short_applies(const FwdArgs& a, int d);
hipError_t launch_fwd_short_bf16(const FwdArgs& a, int d, hipStream_t s);
// phase: -1 = all stages in order, 0 = prepare, 1 = dK/dV/dtable, 2 = dQ.
hipError_t launch_bwd(const BwdArgs& a, int d, bool bf16, int phase, hipStream_t s);
hipError_t launch_dkdv_bf16(const BwdArgs& a, int d, hipStream_t s);
hipError_t launch_dq_bf16(const BwdArgs& a, int d, hipStream_t s);
// Sequences of at most 256 rows (bf16, d <= 32, not a ring step): the whole
// backward (prepare stage, dK, dV, dQ, dtable) in one persistent kernel.
bool bwd_short_applies(const BwdArgs& a, int d);
hipError_t launch_bwd_short_bf16(const BwdArgs& a, int d, hipStream_t s);
hipError_t launch_merge(const MergeArgs& a, bool out_bf16, hipStream_t s);

}  // namespace gt
