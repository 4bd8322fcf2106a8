// Internal declarations shared by the host code and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <unordered_map>
#include <vector>

#include "../../include/actionflow.h"

namespace af {

void set_error(const char* fmt, ...);
void clear_error();

#define AF_HIP(call)                                                                     \
  do {                                                                                   \
    hipError_t e_ = (call);                                                              \
    if (e_ != hipSuccess) {                                                              \
      ::af::set_error("%s failed: %s (%s:%d)", #call, hipGetErrorString(e_), __FILE__, __LINE__); \
      return AF_ERR_DEVICE;                                                              \
    }                                                                                    \
  } while (0)

#define AF_TRY(expr)                \
  do {                              \
    af_status s_ = (expr);          \
    if (s_ != AF_OK) return s_;     \
  } while (0)

inline size_t dtype_size(int dt) { return dt == AF_BF16 ? 2 : 4; }

// ---------------------------------------------------------------- device step descriptor
// Per-call tables the kernels read, uploaded once per call from pinned host memory.
struct DevSeg {            // 8 x int32
  int32_t q_start, q_len, slot, pos0, emit_idx, pad0, pad1, pad2;
};

// ---------------------------------------------------------------- kernel launch arguments
enum Epi { EPI_STORE = 0, EPI_STORE_F32 = 1, EPI_RESID = 2, EPI_SWIGLU = 3, EPI_QKV = 4 };

struct GemmArgs {
  // Activations [M, K]: row-major with row stride lda (fp32), or fragment-tiled (bf16) when
  // astride > 0: 32-row block b at A + b * astride, laid out as frag_off() gives.
  const void* A;
  // Weights, fragment-tiled per column block: bf16 blocks of 32 columns x 16 k (the B operand
  // of the 32x32x16 MFMA), fp32 blocks of 16 columns x 32 k; block nb at B + nb * bstride.
  const void* B;
  int M, N, K, Kp, lda;
  long astride;
  long bstride;
  int splits;      // split-K factor (1 = none)
  float* partial;  // [splits][M][N] fp32 partial sums when splits > 1
  int partials_only;  // with splits > 1: leave the sums and the epilogue to a later kernel
  int col0;        // first column of this launch in the full output (a launch over a column range; unsplit)
  void* out;       // EPI_STORE/_F32/_RESID: [M, N]; EPI_SWIGLU: [M, N/2]; EPI_QKV: queries [M, d_model]
  int ldo;
  long ostride;    // EPI_SWIGLU: > 0 writes the output fragment-tiled (32-row blocks ostride apart)
  const void* resid;  // EPI_RESID: [M, N] (may alias out)
  int ldr;
  // EPI_QKV
  void* ring_k;        // this layer's key region [n_slots][H][max_pos][hd]
  void* ring_v;        // this layer's value region
  const int32_t* row_sp;  // [M][2]: (slot, position) of every packed row
  const float* rope_cs;   // [max_pos][hd/2][2]: (cos, sin)
  int d_model, head_dim, n_heads, max_pos;
};

struct AttnArgs {
  const void* q;   // [M, H*hd] rotated queries
  void* o;         // [M, H*hd]
  const void* ring_k;  // this layer's key region
  const void* ring_v;
  const DevSeg* segs;
  const int32_t* tiles;  // [n_tiles][2]: (segment, first row in segment); multi-row tiles first
  int n_multi;           // tiles of segments with more than one row (the rest are single rows)
  int n_tiles;           // set by the launcher: all tiles
  int n_heads, max_pos, ldq, ldo;  // row strides of q and o (>= H*hd)
  long ostride;              // > 0: o is written fragment-tiled (32-row blocks ostride apart)
  float scale_log2;          // log2(e) / sqrt(hd)
};

hipError_t launch_gemm(int dtype, int epi, const GemmArgs& a, hipStream_t s);
hipError_t launch_attention(int dtype, int head_dim, const AttnArgs& a, int n_tiles, hipStream_t s);
// y row-major (row stride ldy) or, when ystride > 0, fragment-tiled.
hipError_t launch_rmsnorm(int dtype, const void* x, int ldx, const int32_t* rows, const void* g, void* y, int ldy,
                          long ystride, int n_rows, int D, float eps, hipStream_t s);
// Residual update from split-K partial sums followed by the RMSNorm of the updated rows:
// x[m] <- x[m] + sum_s partial[s][m] (rounded as the residual epilogue rounds), then y[m] =
// RMSNorm(x[m]) * g exactly as launch_rmsnorm computes it.  partial is [splits][M][D].
hipError_t launch_resid_norm(int dtype, const float* partial, int splits, void* x, int ldx, const void* g, void* y,
                             int ldy, long ystride, int M, int D, float eps, hipStream_t s);
// Row-major [M, K] (row stride ld) -> fragment-tiled (32-row blocks astride apart), with the
// rows of the last block past M and the columns [K, Kp) written as zeros.
hipError_t launch_to_frag(int dtype, const void* x, int ld, int M, int K, int Kp, void* y, long astride,
                          hipStream_t s);
hipError_t launch_embed(int dtype, const int32_t* ids, const void* table, int vocab, const void* embeds, void* out,
                        int M, int D, int32_t* err_count, hipStream_t s);
hipError_t launch_argmax(const float* logits, int n_rows, int V, int32_t* tokens, hipStream_t s);
// Zero-fills n_runs runs of run_bytes (16-byte multiple, 16-byte aligned), run r at base + r * stride.
hipError_t launch_zero_runs(void* base, int n_runs, size_t stride, size_t run_bytes, hipStream_t s);
// Byte strides of a run copy: run r starts at (r / per_group) * group + (r % per_group) * run.
struct CopyStrides {
  size_t src_group, src_run, dst_group, dst_run;
};
// Copies n_runs runs of run_bytes (16-byte multiple, 16-byte aligned) from src to dst at the
// run offsets of st.  Runs must not overlap one another.
hipError_t launch_copy_runs(const void* src, void* dst, int n_runs, int per_group, const CopyStrides& st,
                            size_t run_bytes, hipStream_t s);
// The same within one buffer: from base + src to base + dst (byte offsets), equal strides.
hipError_t launch_run_copy(void* base, size_t src, size_t dst, int n_runs, int per_group, size_t group_stride,
                           size_t run_stride, size_t run_bytes, hipStream_t s);
// Fragment-tiles N rows of K elements (padded to Kp, a multiple of 32) for the GEMM; srcs is a
// device array of source pointers, map (device, optional) gives (source, row) per output row.
hipError_t launch_frag_pack(int dtype, void* dst, long bstride, const void* const* srcs, const int32_t* map, int N,
                            int K, int Kp, hipStream_t s);
// Padding that keeps concurrently read rows and weight streams off power-of-two strides, so
// they spread over the L2 and HBM channels instead of queueing on one: 128 bytes.
constexpr int STRIDE_PAD_BYTES = 128;
// Columns per packed weight block: 32 for bf16 (32x32x16 MFMA), 16 for fp32 (16x16x4 MFMA).
inline int frag_ncols(int dtype) { return dtype == AF_BF16 ? 32 : 16; }
inline long frag_bstride(int Kp, int dtype) {
  return (long)Kp * frag_ncols(dtype) + STRIDE_PAD_BYTES / (dtype == AF_BF16 ? 2 : 4);
}
// Fragment-tiled activations: one 32-row block holds [Kp/16][64 lanes][8]; lane = row % 32 +
// 32 * ((k % 16) / 8), element k % 8.  Blocks are astride elements apart.
inline long frag_astride(int Kp) { return (long)Kp * 32 + STRIDE_PAD_BYTES / 2; }
__host__ __device__ inline size_t frag_off(int m, int k, long astride) {
  return (size_t)(m >> 5) * astride + (size_t)(k >> 4) * 512 + (size_t)(((m & 31) + ((k >> 3) & 1) * 32) * 8 + (k & 7));
}
int gemm_splits(int dtype, int M, int N, int Kp);  // split-K factor that fills the GPU
int gemm_k_align();                  // K of the packed weights is a multiple of this

constexpr int ATTN_BQ = 64;   // query rows per attention work tile
constexpr int ATTN_WAVES = 8; // waves per attention workgroup (two key groups of four for query tiles)
constexpr int ATTN_BKV = 64;  // keys per LDS tile
constexpr int MAX_SEGMENTS = 4096;

// Which rotary table a caller-free buffer holds: angles pos * theta^(-2j/hd) for rows
// [0, rows) (rows = 0: none).
struct BufferRope {
  float theta = 0.f;
  int head_dim = 0;
  int rows = 0;
};
// af_packed_forward with every device workspace carved from buf (buf_bytes), allocating
// nothing; a step that does not fit is AF_ERR_OUT_OF_RANGE before any launch.
af_status packed_forward_in_buffer(af_weights* w, const int32_t* token_ids, const void* embeds, int32_t M,
                                   const af_segment* segs, int32_t n_seg, af_ring* ring, void* out_hidden,
                                   float* out_logits, int32_t* out_tokens, hipStream_t s, void* buf,
                                   size_t buf_bytes, BufferRope* rope);

}  // namespace af

// ---------------------------------------------------------------- opaque handles
struct af_ring {
  af_ring_desc d;
  void* kv = nullptr;  // device storage, nullptr for a bookkeeping-only ring
  size_t bytes = 0;
  std::vector<int64_t> owner;
  std::vector<int32_t> len;
  int32_t head = 0;
  std::unordered_map<int64_t, int32_t> slot_of;

  size_t slot_stride() const { return (size_t)d.n_kv_heads * d.max_pos * d.head_dim; }
  size_t kv_region() const { return (size_t)d.n_slots * slot_stride(); }
  // element offset of (layer, kv, slot, head, pos)
  size_t offset(int layer, int kv_, int slot, int head, int pos) const {
    return ((((size_t)layer * 2 + kv_) * d.n_slots + slot) * d.n_kv_heads + head) * (size_t)d.max_pos * d.head_dim +
           (size_t)pos * d.head_dim;
  }
};
