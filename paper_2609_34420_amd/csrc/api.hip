// C ABI of libgtattn: host-side validation, then stream-ordered launches.
// Nothing is launched and no output is touched unless every check passes.
#include <cmath>
#include <cstdint>
#include <mutex>

#include "../../include/gt_attn.h"
#include "kernels.hpp"

namespace {

constexpr size_t kAlign = 256;
constexpr int64_t kMaxGrid = 0x7fffffffLL;
// Largest spd row stride (and N): a forward wave reads 64 spd rows through
// one buffer resource whose byte offsets stop at 2^31 - 1, so 64 ld must
// stay below 2^31.
constexpr int64_t kMaxLd = (1LL << 25) - 16;

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

inline bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

inline bool dims_ok(int32_t d) { return d == 8 || d == 16 || d == 32 || d == 64; }

inline bool dtype_ok(gt_dtype_t t) { return t == GT_F32 || t == GT_BF16; }

inline bool scale_ok(float s) { return std::isfinite(s) && s > 0.0f; }

// 16-byte spd loads are legal when every 16-key group of every row starts
// 16-byte aligned.
inline int spd_vec(const uint8_t* spd, int64_t ld, int64_t row_off, int64_t col_off) {
  const uintptr_t base = reinterpret_cast<uintptr_t>(spd) + (uintptr_t)(row_off * ld + col_off);
  return ((base & 15u) == 0 && (ld & 15) == 0) ? 1 : 0;
}

inline gt_status_t launched(hipError_t e) { return e == hipSuccess ? GT_OK : GT_ERR_LAUNCH; }

}  // namespace

extern "C" {

const char* gt_status_string(gt_status_t s) {
  switch (s) {
    case GT_OK: return "GT_OK";
    case GT_ERR_INVALID: return "GT_ERR_INVALID: invalid argument";
    case GT_ERR_UNSUPPORTED: return "GT_ERR_UNSUPPORTED: unsupported head dim or dtype";
    case GT_ERR_WORKSPACE: return "GT_ERR_WORKSPACE: workspace missing or too small";
    case GT_ERR_LAUNCH: return "GT_ERR_LAUNCH: kernel launch failed";
  }
  return "unknown gt_status_t";
}

int32_t gt_attn_version(void) { return 100; }

static gt_status_t ring_impl(const void* q_shard, int64_t Sq, const void* k_shard,
                             const void* v_shard, int64_t Sk, const uint8_t* spd,
                             int64_t ld_spd, int64_t row_off, int64_t col_off,
                             const float* table, int32_t n_buckets, float* o_part,
                             float* lse_part, int32_t H, int32_t d, gt_dtype_t dtype,
                             float scale, void* stream, int32_t accumulate) {
  if (!dtype_ok(dtype)) return GT_ERR_UNSUPPORTED;
  if (!dims_ok(d)) return GT_ERR_UNSUPPORTED;
  if (H < 1 || Sq < 1 || Sk < 0 || row_off < 0 || col_off < 0) return GT_ERR_INVALID;
  if (n_buckets < 1 || n_buckets > 256 || !scale_ok(scale)) return GT_ERR_INVALID;
  if (!q_shard || !table || !o_part || !lse_part) return GT_ERR_INVALID;
  if (Sk > 0 && (!k_shard || !v_shard || !spd)) return GT_ERR_INVALID;
  if (Sk > 0 && ld_spd < col_off + Sk) return GT_ERR_INVALID;
  if (Sk > 0 && ld_spd > kMaxLd) return GT_ERR_UNSUPPORTED;
  if (!aligned16(q_shard) || !aligned16(o_part) || (Sk > 0 && (!aligned16(k_shard) || !aligned16(v_shard))))
    return GT_ERR_INVALID;
  if ((Sq + 127) / 128 * (int64_t)H > kMaxGrid) return GT_ERR_INVALID;
  gt::FwdArgs a{};
  a.q = q_shard; a.k = k_shard; a.v = v_shard;
  a.spd = spd; a.ld_spd = ld_spd; a.row_off = row_off; a.col_off = col_off;
  a.table = table; a.n_buckets = n_buckets;
  a.o = o_part; a.lse = lse_part;
  a.H = H; a.Sq = Sq; a.Sk = Sk; a.scale = scale;
  a.spd_vec = Sk > 0 ? spd_vec(spd, ld_spd, row_off, col_off) : 0;
  a.accumulate = accumulate;
  a.hpb = H; a.spd_bstride = 0;
  return launched(gt::launch_fwd(a, d, dtype == GT_BF16, true, static_cast<hipStream_t>(stream)));
}

gt_status_t gt_attn_ring_step(const void* q_shard, int64_t Sq, const void* k_shard,
                              const void* v_shard, int64_t Sk, const uint8_t* spd,
                              int64_t ld_spd, int64_t row_off, int64_t col_off,
                              const float* table, int32_t n_buckets, float* o_part,
                              float* lse_part, int32_t H, int32_t d, gt_dtype_t dtype,
                              float scale, void* stream) {
  return ring_impl(q_shard, Sq, k_shard, v_shard, Sk, spd, ld_spd, row_off, col_off, table,
                   n_buckets, o_part, lse_part, H, d, dtype, scale, stream, 0);
}

gt_status_t gt_attn_ring_step_acc(const void* q_shard, int64_t Sq, const void* k_shard,
                                  const void* v_shard, int64_t Sk, const uint8_t* spd,
                                  int64_t ld_spd, int64_t row_off, int64_t col_off,
                                  const float* table, int32_t n_buckets, float* o_acc,
                                  float* lse_acc, int32_t H, int32_t d, gt_dtype_t dtype,
                                  float scale, void* stream) {
  return ring_impl(q_shard, Sq, k_shard, v_shard, Sk, spd, ld_spd, row_off, col_off, table,
                   n_buckets, o_acc, lse_acc, H, d, dtype, scale, stream, 1);
}

// B sequences of N nodes, H heads each, run as B * H heads; sequence b reads
// its spd at spd + b * spd_bstride.
static gt_status_t fwd_impl(const void* q, const void* k, const void* v, const uint8_t* spd,
                            int64_t spd_bstride, const float* table, int32_t n_buckets, void* o,
                            float* lse, int32_t B, int32_t H, int64_t N, int32_t d,
                            gt_dtype_t dtype, float scale, void* stream) {
  if (!dtype_ok(dtype)) return GT_ERR_UNSUPPORTED;
  if (!dims_ok(d)) return GT_ERR_UNSUPPORTED;
  if (B < 1 || H < 1 || N < 1 || spd_bstride < 0) return GT_ERR_INVALID;
  if (n_buckets < 1 || n_buckets > 256 || !scale_ok(scale)) return GT_ERR_INVALID;
  if (!q || !k || !v || !spd || !table || !o || !lse) return GT_ERR_INVALID;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o)) return GT_ERR_INVALID;
  const int64_t HT = (int64_t)B * H;
  if (HT > 0x7fffffff || (N + 127) / 128 * HT > kMaxGrid) return GT_ERR_INVALID;
  if (N > kMaxLd) return GT_ERR_UNSUPPORTED;
  gt::FwdArgs a{};
  a.q = q; a.k = k; a.v = v;
  a.spd = spd; a.ld_spd = N; a.row_off = 0; a.col_off = 0;
  a.table = table; a.n_buckets = n_buckets;
  a.o = o; a.lse = lse;
  a.H = (int32_t)HT; a.Sq = N; a.Sk = N; a.scale = scale;
  a.hpb = H; a.spd_bstride = spd_bstride;
  a.spd_vec = spd_vec(spd, N, 0, 0) && spd_bstride % 16 == 0;
  return launched(gt::launch_fwd(a, d, dtype == GT_BF16, dtype == GT_F32, static_cast<hipStream_t>(stream)));
}

gt_status_t gt_attn_fwd(const void* q, const void* k, const void* v, const uint8_t* spd,
                        const float* table, int32_t n_buckets, void* o, float* lse,
                        int32_t H, int64_t N, int32_t d, gt_dtype_t dtype, float scale,
                        void* stream) {
  return fwd_impl(q, k, v, spd, 0, table, n_buckets, o, lse, 1, H, N, d, dtype, scale, stream);
}

gt_status_t gt_attn_fwd_batch(const void* q, const void* k, const void* v, const uint8_t* spd,
                              int64_t spd_bstride, const float* table, int32_t n_buckets, void* o,
                              float* lse, int32_t B, int32_t H, int64_t N, int32_t d,
                              gt_dtype_t dtype, float scale, void* stream) {
  return fwd_impl(q, k, v, spd, spd_bstride, table, n_buckets, o, lse, B, H, N, d, dtype, scale,
                  stream);
}

size_t gt_attn_bwd_workspace_size(int32_t H, int64_t N, int32_t d, gt_dtype_t dtype) {
  (void)d;
  (void)dtype;
  if (H < 1 || N < 1) return 0;
  const size_t rows = (size_t)H * (size_t)N;
  const size_t nblk = (size_t)((N + 255) / 256);
  return 2 * align_up(rows * sizeof(float)) + align_up((size_t)H * nblk * 4 * sizeof(float));
}

static gt_status_t bwd_impl(int32_t phase, const void* q, const void* k, const void* v,
                            const uint8_t* spd, const uint8_t* spd_t, int64_t spd_bstride,
                            const float* table, int32_t n_buckets,
                            const void* o, const float* lse, const void* d_o, void* dq,
                            void* dk, void* dv, float* dtable, void* workspace,
                            size_t workspace_bytes, int32_t B, int32_t Hh, int64_t N, int32_t d,
                            gt_dtype_t dtype, float scale, void* stream) {
  if (!dtype_ok(dtype)) return GT_ERR_UNSUPPORTED;
  if (!dims_ok(d)) return GT_ERR_UNSUPPORTED;
  if (B < 1 || Hh < 1 || N < 1 || spd_bstride < 0) return GT_ERR_INVALID;
  if ((int64_t)B * Hh > 0x7fffffff) return GT_ERR_INVALID;
  const int32_t H = B * Hh;   // heads of the whole batch
  if (n_buckets < 1 || n_buckets > 256 || !scale_ok(scale)) return GT_ERR_INVALID;
  if (!q || !k || !v || !spd || !table || !o || !lse || !d_o || !dq || !dk || !dv || !dtable)
    return GT_ERR_INVALID;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(d_o) ||
      !aligned16(dq) || !aligned16(dk) || !aligned16(dv))
    return GT_ERR_INVALID;
  if ((N + 127) / 128 * (int64_t)H > kMaxGrid) return GT_ERR_INVALID;
  if (N > kMaxLd) return GT_ERR_UNSUPPORTED;
  const size_t need = gt_attn_bwd_workspace_size(H, N, d, dtype);
  if (!workspace || workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return GT_ERR_WORKSPACE;
  const size_t rows = (size_t)H * (size_t)N;
  gt::BwdArgs a{};
  a.q = q; a.k = k; a.v = v;
  a.spd = spd; a.ld_spd = N;
  a.table = table; a.n_buckets = n_buckets;
  a.o = o; a.lse = lse; a.d_o = d_o;
  a.dq = dq; a.dk = dk; a.dv = dv; a.dtable = dtable;
  a.lse2 = static_cast<float*>(workspace);
  a.dlt = reinterpret_cast<float*>(static_cast<char*>(workspace) + align_up(rows * sizeof(float)));
  a.nmax = reinterpret_cast<float*>(static_cast<char*>(workspace) + 2 * align_up(rows * sizeof(float)));
  a.H = H; a.Sq = N; a.Sk = N; a.scale = scale;
  a.row_off = 0; a.col_off = 0; a.accumulate = 0;
  a.hpb = Hh; a.spd_bstride = spd_bstride;
  a.spd_vec = spd_vec(spd, N, 0, 0) && spd_bstride % 16 == 0;
  // The transpose is used only where its rows can be read 16 bytes at a time
  // and one key block's rows (256 of them) stay within 32-bit offsets.
  a.spd_t = (spd_t && spd_vec(spd_t, N, 0, 0) && spd_bstride % 16 == 0 &&
             256 * N < (int64_t(1) << 31)) ? spd_t : nullptr;
  return launched(gt::launch_bwd(a, d, dtype == GT_BF16, phase, static_cast<hipStream_t>(stream)));
}

gt_status_t gt_attn_bwd(const void* q, const void* k, const void* v, const uint8_t* spd,
                        const uint8_t* spd_t, const float* table, int32_t n_buckets, const void* o,
                        const float* lse, const void* d_o, void* dq, void* dk, void* dv,
                        float* dtable, void* workspace, size_t workspace_bytes, int32_t H,
                        int64_t N, int32_t d, gt_dtype_t dtype, float scale, void* stream) {
  return bwd_impl(-1, q, k, v, spd, spd_t, 0, table, n_buckets, o, lse, d_o, dq, dk, dv, dtable,
                  workspace, workspace_bytes, 1, H, N, d, dtype, scale, stream);
}

}  // extern "C"

namespace {

// Device scratch of the allocation-free backward: a file-scope array that
// every GPU the library runs on holds until the process ends. In host code
// the name `scratch` is only a host-side stand-in, never a device address:
// the device address is taken once per device with hipGetSymbolAddress and
// kept in scratch_dev[], and only that pointer is handed to kernels.
constexpr size_t kScratchBytes = size_t(16) << 20;
constexpr int kMaxDevices = 64;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
void* scratch_dev[kMaxDevices];
std::mutex scratch_mu;

// The current device's scratch address (set up on the first call on that
// device, with it current); nullptr if the address cannot be obtained.
void* device_scratch() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (!scratch_dev[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    scratch_dev[dev] = p;
  }
  return scratch_dev[dev];
}

}  // namespace

extern "C" {

size_t gt_attn_bwd_noalloc_max_bytes(void) { return kScratchBytes; }

gt_status_t gt_attn_bwd_noalloc(const void* q, const void* k, const void* v, const uint8_t* spd,
                                const uint8_t* spd_t, const float* table, int32_t n_buckets,
                                const void* o, const float* lse, const void* d_o, void* dq,
                                void* dk, void* dv, float* dtable, int32_t H, int64_t N, int32_t d,
                                gt_dtype_t dtype, float scale, void* stream) {
  // the size limit first: nothing below may allocate
  if (H >= 1 && N >= 1 && gt_attn_bwd_workspace_size(H, N, d, dtype) > kScratchBytes)
    return GT_ERR_WORKSPACE;
  void* ws = device_scratch();
  if (!ws) return GT_ERR_LAUNCH;
  return bwd_impl(-1, q, k, v, spd, spd_t, 0, table, n_buckets, o, lse, d_o, dq, dk, dv, dtable,
                  ws, kScratchBytes, 1, H, N, d, dtype, scale, stream);
}

gt_status_t gt_attn_bwd_batch(const void* q, const void* k, const void* v, const uint8_t* spd,
                              const uint8_t* spd_t, int64_t spd_bstride, const float* table,
                              int32_t n_buckets, const void* o, const float* lse, const void* d_o,
                              void* dq, void* dk, void* dv, float* dtable, void* workspace,
                              size_t workspace_bytes, int32_t B, int32_t H, int64_t N, int32_t d,
                              gt_dtype_t dtype, float scale, void* stream) {
  return bwd_impl(-1, q, k, v, spd, spd_t, spd_bstride, table, n_buckets, o, lse, d_o, dq, dk, dv,
                  dtable, workspace, workspace_bytes, B, H, N, d, dtype, scale, stream);
}

gt_status_t gt_attn_bwd_phase(int32_t phase, const void* q, const void* k, const void* v,
                              const uint8_t* spd, const uint8_t* spd_t, const float* table,
                              int32_t n_buckets,
                              const void* o, const float* lse, const void* d_o, void* dq,
                              void* dk, void* dv, float* dtable, void* workspace,
                              size_t workspace_bytes, int32_t H, int64_t N, int32_t d,
                              gt_dtype_t dtype, float scale, void* stream) {
  if (phase < 0 || phase > 2) return GT_ERR_INVALID;
  return bwd_impl(phase, q, k, v, spd, spd_t, 0, table, n_buckets, o, lse, d_o, dq, dk, dv, dtable,
                  workspace, workspace_bytes, 1, H, N, d, dtype, scale, stream);
}

size_t gt_attn_bwd_ring_workspace_size(int32_t H, int64_t Sq, int64_t Sk, int32_t d,
                                       gt_dtype_t dtype) {
  (void)d;
  (void)dtype;
  if (H < 1 || Sq < 1 || Sk < 0) return 0;
  const size_t rows = (size_t)H * (size_t)Sq;
  const size_t nblk = (size_t)(((Sq > Sk ? Sq : Sk) + 255) / 256);
  return 2 * align_up(rows * sizeof(float)) + align_up((size_t)H * nblk * 4 * sizeof(float));
}

gt_status_t gt_attn_bwd_ring_step(const void* q_shard, const void* o_shard, const float* lse_shard,
                                  const void* d_o_shard, int64_t Sq, const void* k_blk,
                                  const void* v_blk, int64_t Sk, const uint8_t* spd,
                                  int64_t ld_spd, int64_t row_off, int64_t col_off,
                                  const float* table, int32_t n_buckets, float* dq_acc,
                                  float* dk_acc, float* dv_acc, float* dtable_acc,
                                  void* workspace, size_t workspace_bytes, int32_t H, int32_t d,
                                  gt_dtype_t dtype, float scale, void* stream) {
  if (!dtype_ok(dtype)) return GT_ERR_UNSUPPORTED;
  if (!dims_ok(d)) return GT_ERR_UNSUPPORTED;
  if (H < 1 || Sq < 1 || Sk < 0 || row_off < 0 || col_off < 0) return GT_ERR_INVALID;
  if (n_buckets < 1 || n_buckets > 256 || !scale_ok(scale)) return GT_ERR_INVALID;
  if (!q_shard || !o_shard || !lse_shard || !d_o_shard || !table || !dq_acc || !dtable_acc)
    return GT_ERR_INVALID;
  if (Sk > 0 && (!k_blk || !v_blk || !spd || !dk_acc || !dv_acc)) return GT_ERR_INVALID;
  if (Sk > 0 && ld_spd < col_off + Sk) return GT_ERR_INVALID;
  if (Sk > 0 && ld_spd > kMaxLd) return GT_ERR_UNSUPPORTED;
  if (!aligned16(q_shard) || !aligned16(o_shard) || !aligned16(d_o_shard) || !aligned16(dq_acc))
    return GT_ERR_INVALID;
  if (Sk > 0 && (!aligned16(k_blk) || !aligned16(v_blk) || !aligned16(dk_acc) || !aligned16(dv_acc)))
    return GT_ERR_INVALID;
  if (((Sq > Sk ? Sq : Sk) + 127) / 128 * (int64_t)H > kMaxGrid) return GT_ERR_INVALID;
  const size_t need = gt_attn_bwd_ring_workspace_size(H, Sq, Sk, d, dtype);
  if (!workspace || workspace_bytes < need || (reinterpret_cast<uintptr_t>(workspace) % kAlign) != 0)
    return GT_ERR_WORKSPACE;
  if (Sk == 0) return GT_OK;   // an empty key block adds nothing
  const size_t rows = (size_t)H * (size_t)Sq;
  gt::BwdArgs a{};
  a.q = q_shard; a.k = k_blk; a.v = v_blk;
  a.spd = spd; a.spd_t = nullptr; a.ld_spd = ld_spd; a.row_off = row_off; a.col_off = col_off;
  a.table = table; a.n_buckets = n_buckets;
  a.o = o_shard; a.lse = lse_shard; a.d_o = d_o_shard;
  a.dq = dq_acc; a.dk = dk_acc; a.dv = dv_acc; a.dtable = dtable_acc;
  a.lse2 = static_cast<float*>(workspace);
  a.dlt = reinterpret_cast<float*>(static_cast<char*>(workspace) + align_up(rows * sizeof(float)));
  a.nmax = reinterpret_cast<float*>(static_cast<char*>(workspace) + 2 * align_up(rows * sizeof(float)));
  a.hpb = H; a.spd_bstride = 0;
  a.H = H; a.Sq = Sq; a.Sk = Sk; a.scale = scale;
  a.accumulate = 1;
  a.spd_vec = spd_vec(spd, ld_spd, row_off, col_off);
  return launched(gt::launch_bwd(a, d, dtype == GT_BF16, -1, static_cast<hipStream_t>(stream)));
}

gt_status_t gt_attn_merge(const float* o_parts, const float* lse_parts, int32_t n_parts,
                          void* o, float* lse, int32_t H, int64_t S, int32_t d,
                          gt_dtype_t dtype, void* stream) {
  if (!dtype_ok(dtype)) return GT_ERR_UNSUPPORTED;
  if (!dims_ok(d)) return GT_ERR_UNSUPPORTED;
  if (n_parts < 1 || H < 1 || S < 1) return GT_ERR_INVALID;
  if (!o_parts || !lse_parts || !o || !lse) return GT_ERR_INVALID;
  if (!aligned16(o_parts) || !aligned16(o)) return GT_ERR_INVALID;
  const int64_t rows = (int64_t)H * S;
  if ((rows * (d / 4) + 255) / 256 > kMaxGrid) return GT_ERR_INVALID;
  gt::MergeArgs a{};
  a.o_parts = o_parts; a.lse_parts = lse_parts; a.n_parts = n_parts;
  a.o = o; a.lse = lse; a.rows = rows; a.d = d;
  return launched(gt::launch_merge(a, dtype == GT_BF16, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
