// gfx950 kernels of the Cross-Request State Packed Forward.
//
// Every projection is an NT GEMM C[m][n] = sum_k A[m][k] * B[n][k] with A the packed
// activations (M = prefill + decode rows) and B a weight matrix in [out, in] layout, on
// 16x16 MFMA tiles (v_mfma_f32_16x16x32_bf16 for bf16; eight v_mfma_f32_16x16x4f32 for
// fp32), fp32 accumulation, with the step that follows it fused into the epilogue:
//   EPI_QKV     rotary embedding at each row's own position, queries to a buffer, keys and
//               values straight into the row's ring slot (Alg. 2 FusedRoPEAndWriteKV);
//   EPI_RESID   residual add in place (OutputProj and down projection);
//   EPI_SWIGLU  SiLU(gate) * up;
//   EPI_STORE*  plain store (bf16/fp32) and fp32 logits.
// Pairs for the rotary and SwiGLU epilogues: the weights are repacked so that output
// columns come in 16-column blocks [a-block, b-block]; with 16x16 accumulator tiles the
// partner of an element sits in the same lane and register of the next block.
//
// Operand fragments: for both MFMAs a lane (r = lane % 16, g = lane / 16) supplies eight
// consecutive k values, k = 8g .. 8g+7 of a 32-wide k step, for row r of A or column r of
// B; the accumulator tile gives lane (c = lane % 16, g) rows 4g .. 4g+3 of column c.  The
// contraction only needs A and B to use the same lane/element -> k assignment.
#include <hip/hip_runtime.h>

#include "af_internal.h"

namespace af {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(8 * sizeof(float)))) float f32x8;

__device__ __forceinline__ float to_f(bf16 x) { return (float)x; }
__device__ __forceinline__ float to_f(float x) { return x; }
template <typename T>
__device__ __forceinline__ T from_f(float x);
template <>
__device__ __forceinline__ bf16 from_f<bf16>(float x) { return (bf16)x; }
template <>
__device__ __forceinline__ float from_f<float>(float x) { return x; }

// ------------------------------------------------------------------ MFMA per element type
template <typename T>
struct Mma;
template <>
struct Mma<bf16> {
  typedef bf16x8 frag;  // 8 consecutive k, 16 bytes
  __device__ __forceinline__ static f32x4 mma(frag a, frag b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
};
template <>
struct Mma<float> {
  typedef f32x8 frag;  // 8 consecutive k, 32 bytes
  __device__ __forceinline__ static f32x4 mma(frag a, frag b, f32x4 c) {
#pragma unroll
    for (int j = 0; j < 8; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[j], c, 0, 0, 0);
    return c;
  }
};

// 16-byte global/LDS chunk
template <typename T>
struct Chunk {
  static constexpr int N = 16 / sizeof(T);
};

__device__ __forceinline__ uint4 zero4() { return make_uint4(0, 0, 0, 0); }

// ------------------------------------------------------------------ XCD-aware tile order
// Workgroups are dispatched round-robin over the 8 XCDs (each with its own L2).  Give each
// XCD a contiguous run of logical tiles so the M tiles that share a weight panel run on one
// XCD and the panel is fetched from HBM once.
__device__ __forceinline__ int xcd_remap(int bid, int total) {
  const int q = total / 8, r = total % 8;
  const int x = bid % 8, j = bid / 8;
  return x * q + (x < r ? x : r) + j;
}

// ------------------------------------------------------------------ GEMM
template <typename T, int BM, int BN, int WM, int WN, int EPI>
__global__ __launch_bounds__(WM* WN * 64) void gemm_kernel(GemmArgs a) {
  constexpr int NT = WM * WN * 64;
  constexpr int VEC = Chunk<T>::N;               // elements per 16-byte chunk
  constexpr int BK = 128 / sizeof(T);            // 128 bytes of k per row per stage
  constexpr int KSTEPS = BK / 32;                // 32-wide MFMA k steps per stage
  constexpr int LDS_ROW = BK + VEC;              // padded row (elements)
  constexpr int CPR = BK / VEC;                  // chunks per row per stage (= 8)
  constexpr int WTM = BM / WM, WTN = BN / WN;    // wave tile
  constexpr int FM = WTM / 16, FN = WTN / 16;
  constexpr int A_IT = (BM * CPR + NT - 1) / NT;
  constexpr int B_IT = (BN * CPR + NT - 1) / NT;
  static_assert(WTM % 16 == 0 && WTN % 32 == 0, "wave tile: 16-row and 32-column multiples");
  typedef typename Mma<T>::frag frag;

  __shared__ __attribute__((aligned(16))) T As[2][BM * LDS_ROW];
  __shared__ __attribute__((aligned(16))) T Bs[2][BN * LDS_ROW];

  const int n_mt = (a.M + BM - 1) / BM, n_nt = (a.N + BN - 1) / BN;
  const int tile = xcd_remap(blockIdx.x, n_mt * n_nt);
  const int m0 = (tile % n_mt) * BM, n0 = (tile / n_mt) * BN;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm0 = (wave / WN) * WTM, wn0 = (wave % WN) * WTN;
  const int lr = lane & 15, lg = lane >> 4;

  const T* __restrict__ A = (const T*)a.A;
  const T* __restrict__ B = (const T*)a.B;
  const int nk = (a.K + BK - 1) / BK;

  uint4 ra[A_IT], rb[B_IT];
  auto load_stage = [&](int kt) {
    const int k0 = kt * BK;
#pragma unroll
    for (int it = 0; it < A_IT; ++it) {
      const int ci = tid + it * NT;
      const int row = ci / CPR, c = ci % CPR;
      const int gm = m0 + row, gk = k0 + c * VEC;
      ra[it] = (ci < BM * CPR && gm < a.M && gk < a.K) ? *(const uint4*)(A + (size_t)gm * a.lda + gk) : zero4();
    }
#pragma unroll
    for (int it = 0; it < B_IT; ++it) {
      const int ci = tid + it * NT;
      const int row = ci / CPR, c = ci % CPR;
      const int gn = n0 + row, gk = k0 + c * VEC;
      rb[it] = (ci < BN * CPR && gn < a.N && gk < a.K) ? *(const uint4*)(B + (size_t)gn * a.ldb + gk) : zero4();
    }
  };
  auto store_stage = [&](int buf) {
#pragma unroll
    for (int it = 0; it < A_IT; ++it) {
      const int ci = tid + it * NT;
      if (ci < BM * CPR) *(uint4*)(&As[buf][(ci / CPR) * LDS_ROW + (ci % CPR) * VEC]) = ra[it];
    }
#pragma unroll
    for (int it = 0; it < B_IT; ++it) {
      const int ci = tid + it * NT;
      if (ci < BN * CPR) *(uint4*)(&Bs[buf][(ci / CPR) * LDS_ROW + (ci % CPR) * VEC]) = rb[it];
    }
  };

  f32x4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  load_stage(0);
  store_stage(0);
  __syncthreads();

  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_stage(kt + 1);
#pragma unroll
    for (int ks = 0; ks < KSTEPS; ++ks) {
      frag fa[FM], fb[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i)
        fa[i] = *(const frag*)(&As[buf][(wm0 + i * 16 + lr) * LDS_ROW + ks * 32 + lg * 8]);
#pragma unroll
      for (int j = 0; j < FN; ++j)
        fb[j] = *(const frag*)(&Bs[buf][(wn0 + j * 16 + lr) * LDS_ROW + ks * 32 + lg * 8]);
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j) acc[i][j] = Mma<T>::mma(fa[i], fb[j], acc[i][j]);
    }
    if (kt + 1 < nk) store_stage(buf ^ 1);
    __syncthreads();
  }

  // ---------------- epilogue: lane holds rows m0+wm0+16i+4lg+e of column n0+wn0+16j+lr
#pragma unroll
  for (int i = 0; i < FM; ++i) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int m = m0 + wm0 + i * 16 + lg * 4 + e;
      if (m >= a.M) continue;
      if constexpr (EPI == EPI_STORE || EPI == EPI_STORE_F32 || EPI == EPI_RESID) {
#pragma unroll
        for (int j = 0; j < FN; ++j) {
          const int n = n0 + wn0 + j * 16 + lr;
          if (n >= a.N) continue;
          const float v = acc[i][j][e];
          if constexpr (EPI == EPI_STORE) {
            ((T*)a.out)[(size_t)m * a.ldo + n] = from_f<T>(v);
          } else if constexpr (EPI == EPI_STORE_F32) {
            ((float*)a.out)[(size_t)m * a.ldo + n] = v;
          } else {
            const float r = to_f(((const T*)a.resid)[(size_t)m * a.ldr + n]);
            ((T*)a.out)[(size_t)m * a.ldo + n] = from_f<T>(r + v);
          }
        }
      } else {
        // paired epilogues: block j (even) holds the a-halves, block j+1 their partners
#pragma unroll
        for (int j = 0; j < FN; j += 2) {
          const int c = n0 + wn0 + j * 16 + lr;  // column of the a-element, in an even 16-block
          if (c >= a.N) continue;
          const float va = acc[i][j][e], vb = acc[i][j + 1][e];
          if constexpr (EPI == EPI_SWIGLU) {
            const int f = (c >> 5) * 16 + (c & 15);
            const float s = va / (1.0f + __expf(-va));
            ((T*)a.out)[(size_t)m * a.ldo + f] = from_f<T>(s * vb);
          } else {  // EPI_QKV
            const int D = a.d_model, hd = a.head_dim, half = hd >> 1;
            const int region = c / D, cr = c - region * D;
            const int h = cr / hd, jj = cr - h * hd;
            const int dj = (jj >> 5) * 16 + (jj & 15);  // dimension j < hd/2 of this pair
            const int slot = a.row_sp[2 * m], pos = a.row_sp[2 * m + 1];
            if (region == 2) {
              T* dst = (T*)a.ring_v + (((size_t)slot * a.n_heads + h) * a.max_pos + pos) * hd;
              dst[dj] = from_f<T>(va);
              dst[dj + half] = from_f<T>(vb);
            } else {
              const float cs = a.rope_cs[((size_t)pos * half + dj) * 2];
              const float sn = a.rope_cs[((size_t)pos * half + dj) * 2 + 1];
              const float ra_ = va * cs - vb * sn, rb_ = vb * cs + va * sn;
              T* dst = region == 0 ? (T*)a.out + (size_t)m * a.ldo + h * hd
                                   : (T*)a.ring_k + (((size_t)slot * a.n_heads + h) * a.max_pos + pos) * hd;
              dst[dj] = from_f<T>(ra_);
              dst[dj + half] = from_f<T>(rb_);
            }
          }
        }
      }
    }
  }
}

template <typename T, int BM, int BN, int WM, int WN>
static hipError_t gemm_dispatch_epi(int epi, const GemmArgs& a, hipStream_t s) {
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  dim3 grid(tiles), block(WM * WN * 64);
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL((gemm_kernel<T, BM, BN, WM, WN, EPI_STORE>), grid, block, 0, s, a); break;
    case EPI_STORE_F32: hipLaunchKernelGGL((gemm_kernel<T, BM, BN, WM, WN, EPI_STORE_F32>), grid, block, 0, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL((gemm_kernel<T, BM, BN, WM, WN, EPI_RESID>), grid, block, 0, s, a); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm_kernel<T, BM, BN, WM, WN, EPI_SWIGLU>), grid, block, 0, s, a); break;
    case EPI_QKV: hipLaunchKernelGGL((gemm_kernel<T, BM, BN, WM, WN, EPI_QKV>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T>
static hipError_t gemm_dispatch(int epi, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 32) return gemm_dispatch_epi<T, 32, 128, 1, 4>(epi, a, s);
  return gemm_dispatch_epi<T, 96, 128, 2, 2>(epi, a, s);
}

hipError_t launch_gemm(int dtype, int epi, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  return dtype == AF_BF16 ? gemm_dispatch<bf16>(epi, a, s) : gemm_dispatch<float>(epi, a, s);
}

// ------------------------------------------------------------------ segment-aware attention
// One workgroup = one (query tile of <= 64 rows of one segment, head).  Four waves own 16
// query rows each.  Key/value tiles of 64 positions of the segment's ring slot are staged in
// LDS (keys row-major, values transposed).  Scores are computed transposed, S^T = K . Q^T, so
// each lane holds scores of one query and the probabilities feed the P.V MFMA as its B
// operand without a lane exchange; softmax is online in the exp2 domain with the running
// max reduced across the four lanes that share a query.
template <typename T, int HD>
__global__ __launch_bounds__(256) void attention_kernel(AttnArgs a) {
  constexpr int VEC = Chunk<T>::N;
  constexpr int KROW = HD + VEC;            // padded key row (elements)
  constexpr int VROW = ATTN_BKV + VEC;      // padded transposed-value row
  constexpr int KST = HD / 32;              // MFMA k steps over the head dimension
  constexpr int DB = HD / 16;               // 16-dim output blocks
  typedef typename Mma<T>::frag frag;

  __shared__ __attribute__((aligned(16))) T Ks[ATTN_BKV * KROW];
  __shared__ __attribute__((aligned(16))) T Vt[HD * VROW];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int lr = lane & 15, lg = lane >> 4;
  const int seg_i = a.tiles[2 * blockIdx.x], i0 = a.tiles[2 * blockIdx.x + 1];
  const int h = blockIdx.y;
  const DevSeg sg = a.segs[seg_i];
  const int rows_here = min(ATTN_BQ, sg.q_len - i0);
  const int kv_end = sg.pos0 + i0 + rows_here;  // exclusive: keys this tile can see
  const size_t slot_off = ((size_t)sg.slot * a.n_heads + h) * a.max_pos * HD;
  const T* __restrict__ Kg = (const T*)a.ring_k + slot_off;
  const T* __restrict__ Vg = (const T*)a.ring_v + slot_off;

  // this lane's query row (invalid rows are clamped to the last valid one and never stored)
  const int qi = i0 + wave * 16 + lr;
  const bool q_ok = qi < sg.q_len;
  const int qi_c = q_ok ? qi : sg.q_len - 1;
  const int qpos = sg.pos0 + qi_c;
  const int wave_rows = rows_here - wave * 16;  // rows of this wave (<= 0: idle)
  const int wave_last_pos = sg.pos0 + i0 + wave * 16 + min(wave_rows, 16) - 1;

  frag qf[KST];
  {
    const T* qrow = (const T*)a.q + (size_t)(sg.q_start + qi_c) * a.ld + h * HD;
#pragma unroll
    for (int s = 0; s < KST; ++s) qf[s] = *(const frag*)(qrow + s * 32 + lg * 8);
  }

  f32x4 oacc[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d) oacc[d] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  const int n_kt = (kv_end + ATTN_BKV - 1) / ATTN_BKV;
  for (int kt = 0; kt < n_kt; ++kt) {
    const int kb0 = kt * ATTN_BKV;
    // ---- stage keys [kb0, kb0+64) (row-major) and values (transposed) of this slot and head
    constexpr int CPR = HD / VEC;  // chunks per key row
    for (int ci = tid; ci < ATTN_BKV * CPR; ci += 256) {
      const int r = ci / CPR, c = ci % CPR;
      const int key = kb0 + r;
      uint4 kv4 = zero4(), vv4 = zero4();
      if (key < kv_end) {
        kv4 = *(const uint4*)(Kg + (size_t)key * HD + c * VEC);
        vv4 = *(const uint4*)(Vg + (size_t)key * HD + c * VEC);
      }
      *(uint4*)(&Ks[r * KROW + c * VEC]) = kv4;
      T vv[VEC];
      __builtin_memcpy(vv, &vv4, 16);
#pragma unroll
      for (int e = 0; e < VEC; ++e) Vt[(c * VEC + e) * VROW + r] = vv[e];
    }
    __syncthreads();

    if (wave_rows > 0 && kb0 <= wave_last_pos) {
      // ---- S^T = K . Q^T for 4 blocks of 16 keys
      float p[4][4];
      float tmax = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        f32x4 sacc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KST; ++s) {
          const frag kf = *(const frag*)(&Ks[(kb * 16 + lr) * KROW + s * 32 + lg * 8]);
          sacc = Mma<T>::mma(kf, qf[s], sacc);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = kb0 + kb * 16 + lg * 4 + e;
          const float v = key <= qpos ? sacc[e] * a.scale_log2 : -INFINITY;
          p[kb][e] = v;
          tmax = fmaxf(tmax, v);
        }
      }
      tmax = fmaxf(tmax, __shfl_xor(tmax, 16));
      tmax = fmaxf(tmax, __shfl_xor(tmax, 32));
      const float m_new = fmaxf(m_run, tmax);
      const float corr = exp2f(m_run - m_new);  // m_run = -inf on the first tile -> 0
      float psum = 0.f;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float pe = exp2f(p[kb][e] - m_new);
          p[kb][e] = pe;
          psum += pe;
        }
      l_run = l_run * corr + psum;
      m_run = m_new;
#pragma unroll
      for (int d = 0; d < DB; ++d) oacc[d] *= corr;
      // ---- O^T += V^T . P^T over two 32-key chunks.  In bf16 the probabilities are split
      // into a bf16 head and a bf16 remainder (two MFMAs), so P keeps ~16 significant bits and
      // the product is as accurate as an fp32 one; V is exact in bf16.
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        frag pf, pf_lo;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float pv = e < 4 ? p[2 * c][e] : p[2 * c + 1][e - 4];
          pf[e] = from_f<T>(pv);
          pf_lo[e] = from_f<T>(pv - to_f(pf[e]));
        }
#pragma unroll
        for (int d = 0; d < DB; ++d) {
          const T* vrow = &Vt[(d * 16 + lr) * VROW + c * 32 + lg * 4];
          frag vf;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            vf[e] = vrow[e];
            vf[4 + e] = vrow[16 + e];
          }
          oacc[d] = Mma<T>::mma(vf, pf, oacc[d]);
          if constexpr (sizeof(T) == 2) oacc[d] = Mma<T>::mma(vf, pf_lo, oacc[d]);
        }
      }
    }
    __syncthreads();
  }

  if (wave_rows <= 0 || !q_ok) return;
  float l_tot = l_run + __shfl_xor(l_run, 16);
  l_tot += __shfl_xor(l_tot, 32);
  const float inv = 1.0f / l_tot;
  T* orow = (T*)a.o + (size_t)(sg.q_start + qi) * a.ld + h * HD;
#pragma unroll
  for (int d = 0; d < DB; ++d)
#pragma unroll
    for (int e = 0; e < 4; ++e) orow[d * 16 + lg * 4 + e] = from_f<T>(oacc[d][e] * inv);
}

hipError_t launch_attention(int dtype, int head_dim, const AttnArgs& a, int n_tiles, hipStream_t s) {
  if (n_tiles <= 0) return hipSuccess;
  dim3 grid(n_tiles, a.n_heads), block(256);
  if (dtype == AF_BF16) {
    if (head_dim == 128) hipLaunchKernelGGL((attention_kernel<bf16, 128>), grid, block, 0, s, a);
    else if (head_dim == 64) hipLaunchKernelGGL((attention_kernel<bf16, 64>), grid, block, 0, s, a);
    else return hipErrorInvalidValue;
  } else {
    if (head_dim == 128) hipLaunchKernelGGL((attention_kernel<float, 128>), grid, block, 0, s, a);
    else if (head_dim == 64) hipLaunchKernelGGL((attention_kernel<float, 64>), grid, block, 0, s, a);
    else return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------ RMSNorm
// One workgroup of 256 threads per output row; rows[] optionally selects the input row.
template <typename T>
__global__ __launch_bounds__(256) void rmsnorm_kernel(const T* __restrict__ x, int ldx, const int32_t* rows,
                                                      const T* __restrict__ g, T* __restrict__ y, int ldy, int D,
                                                      float eps) {
  __shared__ float red[4];
  const int r_out = blockIdx.x;
  const int r_in = rows ? rows[r_out] : r_out;
  const T* xr = x + (size_t)r_in * ldx;
  float ss = 0.f;
  for (int i = threadIdx.x; i < D; i += 256) {
    const float v = to_f(xr[i]);
    ss += v * v;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  const float tot = red[0] + red[1] + red[2] + red[3];
  const float inv = 1.0f / sqrtf(tot / (float)D + eps);
  T* yr = y + (size_t)r_out * ldy;
  for (int i = threadIdx.x; i < D; i += 256) yr[i] = from_f<T>(to_f(xr[i]) * inv * to_f(g[i]));
}

hipError_t launch_rmsnorm(int dtype, const void* x, int ldx, const int32_t* rows, const void* g, void* y, int ldy,
                          int n_rows, int D, float eps, hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  if (dtype == AF_BF16)
    hipLaunchKernelGGL(rmsnorm_kernel<bf16>, dim3(n_rows), dim3(256), 0, s, (const bf16*)x, ldx, rows,
                       (const bf16*)g, (bf16*)y, ldy, D, eps);
  else
    hipLaunchKernelGGL(rmsnorm_kernel<float>, dim3(n_rows), dim3(256), 0, s, (const float*)x, ldx, rows,
                       (const float*)g, (float*)y, ldy, D, eps);
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
// One workgroup per row; the lowest index among equal maxima wins.
__global__ __launch_bounds__(256) void argmax_kernel(const float* __restrict__ logits, int V, int32_t* tokens) {
  __shared__ float sv[4];
  __shared__ int si[4];
  const float* z = logits + (size_t)blockIdx.x * V;
  float bv = -INFINITY;
  int bi = 0x7fffffff;
  for (int i = threadIdx.x; i < V; i += 256) {
    const float v = z[i];
    if (v > bv) { bv = v; bi = i; }  // strided scan visits indices in increasing order
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
    for (int w = 1; w < 4; ++w)
      if (sv[w] > bv || (sv[w] == bv && si[w] < bi)) { bv = sv[w]; bi = si[w]; }
    tokens[blockIdx.x] = bi == 0x7fffffff ? 0 : bi;
  }
}

hipError_t launch_argmax(const float* logits, int n_rows, int V, int32_t* tokens, hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  hipLaunchKernelGGL(argmax_kernel, dim3(n_rows), dim3(256), 0, s, logits, V, tokens);
  return hipGetLastError();
}

// ------------------------------------------------------------------ weight repacking
// dst row r <- srcs[map[2r]] row map[2r+1]; rows of row_len elements, row_len % (16/size) == 0.
template <typename T>
__global__ __launch_bounds__(256) void copy_rows_kernel(T* __restrict__ dst, const T* const* srcs,
                                                        const int32_t* __restrict__ map, int row_len) {
  const int r = blockIdx.x;
  const T* src = srcs[map[2 * r]] + (size_t)map[2 * r + 1] * row_len;
  T* d = dst + (size_t)r * row_len;
  constexpr int VEC = Chunk<T>::N;
  for (int c = threadIdx.x; c < row_len / VEC; c += 256) ((uint4*)d)[c] = ((const uint4*)src)[c];
}

hipError_t launch_copy_rows(int dtype, void* dst, const void* const* srcs, const int32_t* map, int n_rows,
                            int row_len, hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
  if (dtype == AF_BF16)
    hipLaunchKernelGGL(copy_rows_kernel<bf16>, dim3(n_rows), dim3(256), 0, s, (bf16*)dst, (const bf16* const*)srcs,
                       map, row_len);
  else
    hipLaunchKernelGGL(copy_rows_kernel<float>, dim3(n_rows), dim3(256), 0, s, (float*)dst,
                       (const float* const*)srcs, map, row_len);
  return hipGetLastError();
}

}  // namespace af
