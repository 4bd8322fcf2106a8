// gfx950 kernels beside the projections and the attention: RMSNorm (alone and fused with the
// split-K residual update), the embedding gather, greedy argmax, ring region copies and the
// weight repacking.
#include "af_device.h"

namespace af {

// ------------------------------------------------------------------ RMSNorm
// One workgroup of NORM_THREADS threads per output row (a 4096-wide bf16 row is one 16-byte
// chunk per thread: one memory latency); rows[] optionally selects the input row.  The
// output is row-major (row stride ldy) or, with ystride > 0, fragment-tiled for the GEMM that
// consumes it.  bf16 rows with D % 8 == 0 move 16 bytes per thread access.
constexpr int NORM_THREADS = 512;

// Sum over the workgroup of one value per thread, in a fixed order (lanes by xor shuffles, then
// the waves in order); the same order in every kernel that normalises a row, whose squares are
// accumulated with explicit fused multiply-adds so that every such kernel rounds alike.
__device__ __forceinline__ float norm_block_sum(float v, float* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float tot = red[0];
#pragma unroll
  for (int w = 1; w < NORM_THREADS / 64; ++w) tot += red[w];
  return tot;
}

template <typename T>
__global__ __launch_bounds__(NORM_THREADS) void rmsnorm_kernel(const T* __restrict__ x, int ldx, const int32_t* rows,
                                                      const T* __restrict__ g, T* __restrict__ y, int ldy,
                                                      long ystride, int D, float eps) {
  __shared__ float red[NORM_THREADS / 64];
  const int r_out = blockIdx.x;
  const int r_in = rows ? rows[r_out] : r_out;
  const T* xr = x + (size_t)r_in * ldx;
  constexpr int V = 16 / sizeof(T);
  const bool vec = sizeof(T) == 2 && D % 8 == 0 && ldx % 8 == 0;
  float ss = 0.f;
  if (vec && D <= NORM_THREADS * V) {
    // at most one chunk per thread: the row and the gain are loaded at once and the row stays in
    // registers for the normalisation; the same arithmetic, in the same order, as below
    const int i = threadIdx.x * V;
    const bool has = i < D;
    T v[V], gv[V];
    if (has) {
      *(uint4*)v = *(const uint4*)(xr + i);
      *(uint4*)gv = *(const uint4*)(g + i);
#pragma unroll
      for (int e = 0; e < V; ++e) ss = fmaf(to_f(v[e]), to_f(v[e]), ss);
    }
    const float tot = norm_block_sum(ss, red);
    const float inv = 1.0f / sqrtf(tot / (float)D + eps);
    if (has) {
      T o[V];
#pragma unroll
      for (int e = 0; e < V; ++e) o[e] = from_f<T>(to_f(v[e]) * inv * to_f(gv[e]));
      T* dst = ystride > 0 ? y + frag_off(r_out, i, ystride) : y + (size_t)r_out * ldy + i;
      *(uint4*)dst = *(const uint4*)o;
    }
    return;
  }
  if (vec) {
    for (int i = threadIdx.x * V; i < D; i += NORM_THREADS * V) {
      T v[V];
      *(uint4*)v = *(const uint4*)(xr + i);
#pragma unroll
      for (int e = 0; e < V; ++e) ss = fmaf(to_f(v[e]), to_f(v[e]), ss);
    }
  } else {
    for (int i = threadIdx.x; i < D; i += NORM_THREADS) {
      const float v = to_f(xr[i]);
      ss = fmaf(v, v, ss);
    }
  }
  const float tot = norm_block_sum(ss, red);
  const float inv = 1.0f / sqrtf(tot / (float)D + eps);
  if (vec) {
    for (int i = threadIdx.x * V; i < D; i += NORM_THREADS * V) {
      T v[V], gv[V], o[V];
      *(uint4*)v = *(const uint4*)(xr + i);
      *(uint4*)gv = *(const uint4*)(g + i);
#pragma unroll
      for (int e = 0; e < V; ++e) o[e] = from_f<T>(to_f(v[e]) * inv * to_f(gv[e]));
      T* dst = ystride > 0 ? y + frag_off(r_out, i, ystride) : y + (size_t)r_out * ldy + i;
      *(uint4*)dst = *(const uint4*)o;
    }
  } else {
    for (int i = threadIdx.x; i < D; i += NORM_THREADS) {
      const T o = from_f<T>(to_f(xr[i]) * inv * to_f(g[i]));
      y[ystride > 0 ? frag_off(r_out, i, ystride) : (size_t)r_out * ldy + i] = o;
    }
  }
}

// Many rows of width D <= 4096 (bf16): one wave per row, eight rows per workgroup.  The gain is
// loaded once per workgroup into LDS instead of once per row, every chunk of the row is
// requested before any is used and stays in registers, and no workgroup barrier sits between
// a row's load and its store.  Lane l holds chunks l + 64 i, which are the chunks thread
// 64 i + l of rmsnorm_kernel holds; its squares are summed, tree-reduced over the 64 lanes and
// the eight partial sums added in the same order as there, so every output is bit-identical.
constexpr int NORM_ROWS_PER_WG = 8;
__global__ __launch_bounds__(64 * NORM_ROWS_PER_WG) void rmsnorm_rows_kernel(const bf16* __restrict__ x, int ldx,
                                                                       const int32_t* rows,
                                                                       const bf16* __restrict__ g, bf16* __restrict__ y,
                                                                       int ldy, long ystride, int n_rows, int D,
                                                                       float eps) {
  constexpr int CPL = NORM_THREADS / 64;  // chunks per lane: 4096 / 8 / 64
  static_assert(NORM_THREADS == 64 * NORM_ROWS_PER_WG, "one thread of rmsnorm_kernel per chunk");
  __shared__ __attribute__((aligned(16))) bf16 gs[NORM_THREADS * 8];
  const int lane = threadIdx.x & 63, r = blockIdx.x * NORM_ROWS_PER_WG + (threadIdx.x >> 6);
  const int n_chunks = D / 8;
  if ((int)threadIdx.x < n_chunks) *(uint4*)&gs[8 * threadIdx.x] = *(const uint4*)(g + 8 * threadIdx.x);
  bf16 v[CPL][8];
  const bf16* xr = x + (size_t)(r < n_rows ? (rows ? rows[r] : r) : 0) * ldx;
#pragma unroll
  for (int i = 0; i < CPL; ++i)
    if (64 * i + lane < n_chunks && r < n_rows) *(uint4*)v[i] = *(const uint4*)(xr + 8 * (64 * i + lane));
  float tot = 0.f;
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    float ss = 0.f;
    if (64 * i + lane < n_chunks && r < n_rows)
#pragma unroll
      for (int e = 0; e < 8; ++e) ss = fmaf(to_f(v[i][e]), to_f(v[i][e]), ss);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
    tot = i == 0 ? ss : tot + ss;
  }
  const float inv = 1.0f / sqrtf(tot / (float)D + eps);
  __syncthreads();  // the gain is in LDS
  if (r >= n_rows) return;
#pragma unroll
  for (int i = 0; i < CPL; ++i) {
    const int c = 64 * i + lane;
    if (c >= n_chunks) continue;
    bf16 gv[8], o[8];
    *(uint4*)gv = *(const uint4*)&gs[8 * c];
#pragma unroll
    for (int e = 0; e < 8; ++e) o[e] = from_f<bf16>(to_f(v[i][e]) * inv * to_f(gv[e]));
    bf16* dst = ystride > 0 ? y + frag_off(r, 8 * c, ystride) : y + (size_t)r * ldy + 8 * c;
    *(uint4*)dst = *(const uint4*)o;
  }
}

// Rows per launch from which the row-per-wave kernel is used (its workgroups then still number
// 128 or more).
constexpr int NORM_ROWS_MIN = 1024;

hipError_t launch_rmsnorm(int dtype, const void* x, int ldx, const int32_t* rows, const void* g, void* y, int ldy,
                          long ystride, int n_rows, int D, float eps, hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  if (dtype == AF_BF16 && n_rows >= NORM_ROWS_MIN && D % 8 == 0 && D <= 8 * NORM_THREADS && ldx % 8 == 0) {
    hipLaunchKernelGGL(rmsnorm_rows_kernel, dim3((n_rows + NORM_ROWS_PER_WG - 1) / NORM_ROWS_PER_WG),
                       dim3(64 * NORM_ROWS_PER_WG), 0, s, (const bf16*)x, ldx, rows, (const bf16*)g, (bf16*)y, ldy,
                       ystride, n_rows, D, eps);
    return hipGetLastError();
  }
  if (dtype == AF_BF16)
    hipLaunchKernelGGL(rmsnorm_kernel<bf16>, dim3(n_rows), dim3(NORM_THREADS), 0, s, (const bf16*)x, ldx, rows,
                       (const bf16*)g, (bf16*)y, ldy, ystride, D, eps);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(n_rows), dim3(NORM_THREADS), 0, s, (const float*)x, ldx, rows,
                       (const float*)g, (float*)y, ldy, ystride, D, eps);
  return hipGetLastError();
}

// Split-K sum + residual + RMSNorm, one workgroup per row.  Each thread covers the same
// elements, in the same order, as splitk_reduce_kernel<EPI_RESID> followed by rmsnorm_kernel
// would, so the residual row and the normalised row are bit-identical to that pair of launches
// (one launch fewer, and the row is summed and normalised while it is on chip).
template <typename T>
__global__ __launch_bounds__(NORM_THREADS) void resid_norm_kernel(const float* __restrict__ partial, int splits, T* x, int ldx,
                                                         const T* __restrict__ g, T* __restrict__ y, int ldy,
                                                         long ystride, int M, int D, float eps) {
  __shared__ float red[NORM_THREADS / 64];
  const int m = blockIdx.x;
  T* xr = x + (size_t)m * ldx;
  const size_t plane = (size_t)M * D;
  constexpr int V = 16 / sizeof(T);
  const bool vec = sizeof(T) == 2 && D % 8 == 0 && ldx % 8 == 0;
  float ss = 0.f;
  if (vec && D <= NORM_THREADS * V) {
    // at most one chunk per thread: every load (the partial sums of all splits, the residual
    // row, the gain) is issued before anything waits, and the updated residual stays in
    // registers for the normalisation; the same arithmetic, in the same order, as below
    const int i = threadIdx.x * V;
    const bool has = i < D;
    constexpr int MAXS = 8;
    float t[MAXS][8];
    T res[8], gv[8];
    if (has) {
#pragma unroll
      for (int sp = 0; sp < MAXS; ++sp)
        if (sp < splits) load8<float>(partial + sp * plane + (size_t)m * D + i, t[sp]);
      load8<T>(xr + i, res);
      load8<T>(g + i, gv);
    }
    T r[8];
    if (has) {
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = 0.f;
#pragma unroll
      for (int sp = 0; sp < MAXS; ++sp)
        if (sp < splits)
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] += t[sp][e];
      for (int sp = MAXS; sp < splits; ++sp) {
        float u[8];
        load8<float>(partial + sp * plane + (size_t)m * D + i, u);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] += u[e];
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) r[e] = from_f<T>(to_f(res[e]) + v[e]);
      store8<T>(xr + i, r);
#pragma unroll
      for (int e = 0; e < 8; ++e) ss = fmaf(to_f(r[e]), to_f(r[e]), ss);
    }
    const float tot = norm_block_sum(ss, red);
    const float inv = 1.0f / sqrtf(tot / (float)D + eps);
    if (has) {
      T o[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) o[e] = from_f<T>(to_f(r[e]) * inv * to_f(gv[e]));
      T* dst = ystride > 0 ? y + frag_off(m, i, ystride) : y + (size_t)m * ldy + i;
      *(uint4*)dst = *(const uint4*)o;
    }
    return;
  }
  if (vec) {
    for (int i = threadIdx.x * V; i < D; i += NORM_THREADS * V) {
      // all of this chunk's partial sums are requested before any is added (one memory latency
      // instead of one per split); they are added in split order
      constexpr int MAXS = 8;
      float t[MAXS][8];
#pragma unroll
      for (int sp = 0; sp < MAXS; ++sp)
        if (sp < splits) load8<float>(partial + sp * plane + (size_t)m * D + i, t[sp]);
      float v[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = 0.f;
#pragma unroll
      for (int sp = 0; sp < MAXS; ++sp)
        if (sp < splits)
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] += t[sp][e];
      for (int sp = MAXS; sp < splits; ++sp) {
        float u[8];
        load8<float>(partial + sp * plane + (size_t)m * D + i, u);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] += u[e];
      }
      T res[8], r[8];
      load8<T>(xr + i, res);
#pragma unroll
      for (int e = 0; e < 8; ++e) r[e] = from_f<T>(to_f(res[e]) + v[e]);
      store8<T>(xr + i, r);
#pragma unroll
      for (int e = 0; e < 8; ++e) ss = fmaf(to_f(r[e]), to_f(r[e]), ss);
    }
  } else {
    for (int i = threadIdx.x; i < D; i += NORM_THREADS) {
      float v = 0.f;
      for (int sp = 0; sp < splits; ++sp) v += partial[sp * plane + (size_t)m * D + i];
      const T r = from_f<T>(to_f(xr[i]) + v);
      xr[i] = r;
      ss = fmaf(to_f(r), to_f(r), ss);
    }
  }
  const float tot = norm_block_sum(ss, red);
  const float inv = 1.0f / sqrtf(tot / (float)D + eps);
  if (vec) {  // each thread re-reads only the elements it wrote
    for (int i = threadIdx.x * V; i < D; i += NORM_THREADS * V) {
      T v[V], gv[V], o[V];
      *(uint4*)v = *(const uint4*)(xr + i);
      *(uint4*)gv = *(const uint4*)(g + i);
#pragma unroll
      for (int e = 0; e < V; ++e) o[e] = from_f<T>(to_f(v[e]) * inv * to_f(gv[e]));
      T* dst = ystride > 0 ? y + frag_off(m, i, ystride) : y + (size_t)m * ldy + i;
      *(uint4*)dst = *(const uint4*)o;
    }
  } else {
    for (int i = threadIdx.x; i < D; i += NORM_THREADS) {
      const T o = from_f<T>(to_f(xr[i]) * inv * to_f(g[i]));
      y[ystride > 0 ? frag_off(m, i, ystride) : (size_t)m * ldy + i] = o;
    }
  }
}

hipError_t launch_resid_norm(int dtype, const float* partial, int splits, void* x, int ldx, const void* g, void* y,
                             int ldy, long ystride, int M, int D, float eps, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (splits < 1 || !partial) return hipErrorInvalidValue;
  if (dtype == AF_BF16)
    hipLaunchKernelGGL(resid_norm_kernel<bf16>, dim3(M), dim3(NORM_THREADS), 0, s, partial, splits, (bf16*)x, ldx,
                       (const bf16*)g, (bf16*)y, ldy, ystride, M, D, eps);
  else
    hipLaunchKernelGGL(resid_norm_kernel<float>, dim3(M), dim3(NORM_THREADS), 0, s, partial, splits, (float*)x, ldx,
                       (const float*)g, (float*)y, ldy, ystride, M, D, eps);
  return hipGetLastError();
}

// Row-major -> fragment-tiled copy; one thread per 8 consecutive k of one row.
__global__ __launch_bounds__(256) void to_frag_kernel(const bf16* __restrict__ x, int ld, int M, int K, int Kp,
                                                      bf16* __restrict__ y, long astride, int rows_padded) {
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  const int groups = Kp / 8;
  if (idx >= (size_t)rows_padded * groups) return;
  const int m = (int)(idx / groups), k0 = (int)(idx % groups) * 8;
  bf16 v[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] = (m < M && k0 + e < K) ? x[(size_t)m * ld + k0 + e] : (bf16)0.f;
  *(uint4*)(y + frag_off(m, k0, astride)) = *(const uint4*)v;
}

hipError_t launch_to_frag(int dtype, const void* x, int ld, int M, int K, int Kp, void* y, long astride,
                          hipStream_t s) {
  if (dtype != AF_BF16 || M <= 0 || K <= 0 || Kp < K || Kp % 16 || astride < (long)Kp * 32) return hipErrorInvalidValue;
  const int rows_padded = (M + 31) / 32 * 32;
  const size_t n = (size_t)rows_padded * (Kp / 8);
  hipLaunchKernelGGL(to_frag_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, (const bf16*)x, ld, M, K, Kp,
                     (bf16*)y, astride, rows_padded);
  return hipGetLastError();
}

// ------------------------------------------------------------------ embedding gather
template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(const int32_t* __restrict__ ids, const T* __restrict__ table,
                                                    int vocab, const T* __restrict__ embeds, T* __restrict__ out,
                                                    int D, int32_t* err_count) {
  const int m = blockIdx.x;
  const int id = ids[m];
  const T* src = nullptr;
  if (id >= 0 && id < vocab) src = table + (size_t)id * D;
  else if (id == -1 && embeds) src = embeds + (size_t)m * D;
  if (!src && threadIdx.x == 0) atomicAdd(err_count, 1);
  T* dst = out + (size_t)m * D;
  constexpr int V = 16 / sizeof(T);
  if (D % V == 0 && (((uintptr_t)dst | (uintptr_t)src) & 15) == 0) {  // 16-byte chunks
    for (int i = threadIdx.x * V; i < D; i += 256 * V) *(uint4*)(dst + i) = src ? *(const uint4*)(src + i) : zero4();
    return;
  }
  for (int i = threadIdx.x; i < D; i += 256) dst[i] = src ? src[i] : from_f<T>(0.f);
}

hipError_t launch_embed(int dtype, const int32_t* ids, const void* table, int vocab, const void* embeds, void* out,
                        int M, int D, int32_t* err_count, hipStream_t s) {
  if (M <= 0) return hipSuccess;
  if (dtype == AF_BF16)
    hipLaunchKernelGGL(embed_kernel<bf16>, dim3(M), dim3(256), 0, s, ids, (const bf16*)table, vocab,
                       (const bf16*)embeds, (bf16*)out, D, err_count);
  else
    hipLaunchKernelGGL(embed_kernel<float>, dim3(M), dim3(256), 0, s, ids, (const float*)table, vocab,
                       (const float*)embeds, (float*)out, D, err_count);
  return hipGetLastError();
}

// ------------------------------------------------------------------ greedy argmax
// One workgroup of 1024 threads per row, 16-byte loads; the lowest index among equal maxima wins
// (each thread scans its indices in increasing order and keeps the first maximum it meets; the
// reduction prefers the lower index on equal values).
__global__ __launch_bounds__(1024) void argmax_kernel(const float* __restrict__ logits, int V, int32_t* tokens) {
  __shared__ float sv[16];
  __shared__ int si[16];
  const float* z = logits + (size_t)blockIdx.x * V;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  if (V % 4 == 0 && ((uintptr_t)z & 15) == 0) {
    const float4* z4 = (const float4*)z;
    for (int i = threadIdx.x; i < V / 4; i += 1024) {
      const float4 v = z4[i];
      if (v.x > bv) { bv = v.x; bi = 4 * i; }
      if (v.y > bv) { bv = v.y; bi = 4 * i + 1; }
      if (v.z > bv) { bv = v.z; bi = 4 * i + 2; }
      if (v.w > bv) { bv = v.w; bi = 4 * i + 3; }
    }
  } else {
    for (int i = threadIdx.x; i < V; i += 1024) {
      const float v = z[i];
      if (v > bv) { bv = v; bi = i; }
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const float ov = __shfl_xor(bv, o);
    const int oi = __shfl_xor(bi, o);
    if (ov > bv || (ov == bv && oi < bi)) { bv = ov; bi = oi; }
  }
  if ((threadIdx.x & 63) == 0) { sv[threadIdx.x >> 6] = bv; si[threadIdx.x >> 6] = bi; }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 16; ++w)
      if (sv[w] > bv || (sv[w] == bv && si[w] < bi)) { bv = sv[w]; bi = si[w]; }
    tokens[blockIdx.x] = bi == 0x7fffffff ? 0 : bi;
  }
}

hipError_t launch_argmax(const float* logits, int n_rows, int V, int32_t* tokens, hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(argmax_kernel, dim3(n_rows), dim3(1024), 0, s, logits, V, tokens);
  return hipGetLastError();
}

// ------------------------------------------------------------------ ring region copies
// Stage moves and copies between rings: 16-byte copies, one workgroup per 64 KiB of a run.
__global__ __launch_bounds__(256) void run_copy_kernel(const char* src, char* dst, int per_group, CopyStrides st,
                                                       size_t run_bytes) {
  const int r = blockIdx.x;
  const size_t g = (size_t)(r / per_group), h = (size_t)(r % per_group);
  const uint4* from = (const uint4*)(src + g * st.src_group + h * st.src_run);
  uint4* to = (uint4*)(dst + g * st.dst_group + h * st.dst_run);
  const size_t n16 = run_bytes / 16, chunk = (size_t)blockIdx.y * 4096;  // 64 KiB per block
  const size_t end = n16 < chunk + 4096 ? n16 : chunk + 4096;
  for (size_t i = chunk + threadIdx.x; i < end; i += 256) to[i] = from[i];
}

hipError_t launch_copy_runs(const void* src, void* dst, int n_runs, int per_group, const CopyStrides& st,
                            size_t run_bytes, hipStream_t s) {
  if (n_runs <= 0 || run_bytes == 0) return hipSuccess;
  if (run_bytes % 16 || (uintptr_t)src % 16 || (uintptr_t)dst % 16 || st.src_group % 16 || st.src_run % 16 ||
      st.dst_group % 16 || st.dst_run % 16 || per_group <= 0)
    return hipErrorInvalidValue;
  const size_t chunks = (run_bytes / 16 + 4095) / 4096;
  if (chunks > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(run_copy_kernel, dim3(n_runs, (unsigned)chunks), dim3(256), 0, s, (const char*)src, (char*)dst,
                     per_group, st, run_bytes);
  return hipGetLastError();
}

hipError_t launch_run_copy(void* base, size_t src, size_t dst, int n_runs, int per_group, size_t group_stride,
                           size_t run_stride, size_t run_bytes, hipStream_t s) {
  const CopyStrides st{group_stride, run_stride, group_stride, run_stride};
  return launch_copy_runs((const char*)base + src, (char*)base + dst, n_runs, per_group, st, run_bytes, s);
}

__global__ __launch_bounds__(256) void zero_runs_kernel(char* base, size_t stride, size_t run_bytes) {
  uint4* p = (uint4*)(base + (size_t)blockIdx.x * stride);
  const size_t n16 = run_bytes / 16, chunk = (size_t)blockIdx.y * 4096;  // 64 KiB per block
  const size_t end = n16 < chunk + 4096 ? n16 : chunk + 4096;
  for (size_t i = chunk + threadIdx.x; i < end; i += 256) p[i] = zero4();
}

hipError_t launch_zero_runs(void* base, int n_runs, size_t stride, size_t run_bytes, hipStream_t s) {
  if (n_runs <= 0 || run_bytes == 0) return hipSuccess;
  if (run_bytes % 16 || (uintptr_t)base % 16 || stride % 16) return hipErrorInvalidValue;
  const size_t chunks = (run_bytes / 16 + 4095) / 4096;
  if (chunks > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(zero_runs_kernel, dim3(n_runs, (unsigned)chunks), dim3(256), 0, s, (char*)base, stride,
                     run_bytes);
  return hipGetLastError();
}

// ------------------------------------------------------------------ weight repacking
// dst: fragment-tiled [N/16][Kp/32][64 lanes][8] (see the GEMM); source row n is
// srcs[map[2n]] row map[2n+1] (or src0 row n without a map), rows of K elements, k >= K zero.
// Weight packing.  bf16: block (nb, k16) of 32 columns x 16 k, lane l -> column 32 nb + l % 32,
// k = 16 k16 + 8 (l / 32) + e (the B operand of the 32x32x16 MFMA).  fp32: block (nb, k32) of 16
// columns x 32 k, lane l -> column 16 nb + l % 16, k = 32 k32 + 8 (l / 16) + e.  Columns >= N
// and k >= K are zero.
template <typename T, int NC>
__global__ __launch_bounds__(256) void frag_pack_kernel(T* __restrict__ dst, long bstride, const T* const* srcs,
                                                        const int32_t* __restrict__ map, int N, int K, int Kp) {
  constexpr int KB = 512 / NC;  // k per block
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  const int ksteps = Kp / KB, n_blocks = (N + NC - 1) / NC;
  const size_t total = (size_t)n_blocks * ksteps * 64;
  if (idx >= total) return;
  const int lane = (int)(idx & 63);
  const size_t blk = idx >> 6;
  const int ks = (int)(blk % ksteps), nb = (int)(blk / ksteps);
  const int n = nb * NC + lane % NC, k0 = ks * KB + 8 * (lane / NC);
  T* d = dst + (size_t)nb * bstride + ((size_t)ks * 64 + lane) * 8;
  if (n >= N) {
#pragma unroll
    for (int e = 0; e < 8; ++e) d[e] = from_f<T>(0.f);
    return;
  }
  const T* src = map ? srcs[map[2 * n]] + (size_t)map[2 * n + 1] * K : srcs[0] + (size_t)n * K;
#pragma unroll
  for (int e = 0; e < 8; ++e) d[e] = k0 + e < K ? src[k0 + e] : from_f<T>(0.f);
}

hipError_t launch_frag_pack(int dtype, void* dst, long bstride, const void* const* srcs, const int32_t* map, int N,
                            int K, int Kp, hipStream_t s) {
  const int nc = frag_ncols(dtype);
  if (N <= 0 || N % 16 || Kp % 32 || Kp < K || bstride < (long)Kp * nc) return hipErrorInvalidValue;
  const size_t total = (size_t)((N + nc - 1) / nc) * (Kp * nc / 512) * 64;
  dim3 grid((unsigned)((total + 255) / 256)), block(256);
  if (dtype == AF_BF16)
    hipLaunchKernelGGL((frag_pack_kernel<bf16, 32>), grid, block, 0, s, (bf16*)dst, bstride,
                       (const bf16* const*)srcs, map, N, K, Kp);
  else
    hipLaunchKernelGGL((frag_pack_kernel<float, 16>), grid, block, 0, s, (float*)dst, bstride,
                       (const float* const*)srcs, map, N, K, Kp);
  return hipGetLastError();
}

}  // namespace af
