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
  const void* A;  // [M, K] activations, row stride lda elements
  const void* B;  // weights, fragment-tiled: n-block nb at B + nb * bstride, [Kp/32][64][8] each
  int M, N, K, Kp, lda;
  long bstride;    // elements between consecutive 16-column blocks (>= Kp * 16, padded)
  int splits;      // split-K factor (1 = none)
  float* partial;  // [splits][M][N] fp32 partial sums when splits > 1
  void* out;       // EPI_STORE/_F32/_RESID: [M, N]; EPI_SWIGLU: [M, N/2]; EPI_QKV: queries [M, d_model]
  int ldo;
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
  const int32_t* tiles;  // [n_tiles][2]: (segment, first row in segment)
  int n_heads, max_pos, ldq, ldo;  // row strides of q and o (>= H*hd)
  float scale_log2;          // log2(e) / sqrt(hd)
};

hipError_t launch_gemm(int dtype, int epi, const GemmArgs& a, hipStream_t s);
hipError_t launch_attention(int dtype, int head_dim, const AttnArgs& a, int n_tiles, hipStream_t s);
hipError_t launch_rmsnorm(int dtype, const void* x, int ldx, const int32_t* rows, const void* g, void* y, int ldy,
                          int n_rows, int D, float eps, hipStream_t s);
hipError_t launch_embed(int dtype, const int32_t* ids, const void* table, int vocab, const void* embeds, void* out,
                        int M, int D, int32_t* err_count, hipStream_t s);
hipError_t launch_argmax(const float* logits, int n_rows, int V, int32_t* tokens, hipStream_t s);
// Fragment-tiles N rows of K elements (padded to Kp, a multiple of 32) for the GEMM; srcs is a
// device array of source pointers, map (device, optional) gives (source, row) per output row.
hipError_t launch_frag_pack(int dtype, void* dst, long bstride, const void* const* srcs, const int32_t* map, int N,
                            int K, int Kp, hipStream_t s);
// Padding that keeps concurrently read rows and weight streams off power-of-two strides, so
// they spread over the L2 and HBM channels instead of queueing on one: 128 bytes.
constexpr int STRIDE_PAD_BYTES = 128;
inline long frag_bstride(int Kp, int dtype) { return (long)Kp * 16 + STRIDE_PAD_BYTES / (dtype == AF_BF16 ? 2 : 4); }
int gemm_block_m(int dtype, int M);  // rows per GEMM workgroup tile for M packed rows
int gemm_block_n();                  // columns per GEMM workgroup tile
int gemm_k_align();                  // K of the packed weights is a multiple of this

constexpr int ATTN_BQ = 64;   // query rows per attention work tile
constexpr int ATTN_BKV = 64;  // keys per LDS tile
constexpr int MAX_SEGMENTS = 4096;

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
