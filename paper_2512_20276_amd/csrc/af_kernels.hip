// gfx950 kernels of the Cross-Request State Packed Forward.
//
// Every projection is an NT GEMM C[m][n] = sum_k A[m][k] * B[n][k] with A the packed
// activations (M = prefill + decode rows) and B a weight matrix in [out, in] layout, with fp32
// accumulation and the step that follows it fused into the epilogue:
//   EPI_QKV     rotary embedding at each row's own position, queries to a buffer, keys and
//               values straight into the row's ring slot (Alg. 2 FusedRoPEAndWriteKV);
//   EPI_RESID   residual add in place (OutputProj and down projection);
//   EPI_SWIGLU  SiLU(gate) * up;
//   EPI_STORE*  plain store (bf16/fp32) and fp32 logits.
// bf16 runs on v_mfma_f32_32x32x16_bf16 (gemm32_kernel) with both operands fragment-tiled in
// HBM; fp32 (small models) on v_mfma_f32_16x16x4f32 with row-major activations (gemm_kernel).
// Pairs for the rotary and SwiGLU epilogues: the weights are repacked so that each 16-column
// group holds 8 a-columns and then their 8 partners; in either accumulator layout the partner
// of lane l's element is lane l ^ 8's, one lane exchange away.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <type_traits>

#include "af_internal.h"

namespace af {

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(8 * sizeof(float)))) float f32x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(unsigned)))) unsigned u32x4;  // raw 16 bytes

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

// Compile-time loop: f(std::integral_constant<int, I>) for I in [B, E).  Register arrays indexed
// by such constants are promoted to registers before any loop transformation runs.
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// ------------------------------------------------------------------ XCD-aware tile order
// Workgroups are dispatched round-robin over the 8 XCDs (each with its own L2).  Give each
// XCD a contiguous run of logical tiles so the M tiles that share a weight panel run on one
// XCD and the panel is fetched from HBM once.
#ifndef AF_XCD_REMAP
#define AF_XCD_REMAP 1
#endif
__device__ __forceinline__ int xcd_remap(int bid, int total) {
  if (!AF_XCD_REMAP) return bid;
  const int q = total / 8, r = total % 8;
  const int x = bid % 8, j = bid / 8;
  return x * q + (x < r ? x : r) + j;
}

// ------------------------------------------------------------------ GEMM
// Weights are stored fragment-tiled: block (n_blk, k_step) of 16 output columns x 32 k is
// 64 lanes x 8 elements, contiguous, in exactly the order the MFMA B operand wants it, so
// each wave streams its weight fragments from HBM straight into registers (one coalesced
// 1 KB load per block for bf16) through a ring PF k-steps deep.  The activations, shared by
// the four waves of a workgroup, go through LDS in the same fragment order (conflict-free
// 16-byte reads), double-buffered per 128-byte k stage.  A workgroup covers BM rows x
// 4 * WTN columns; split-K workgroups write fp32 partial tiles that a second kernel sums in
// split order (deterministic) before the epilogue.
template <typename T, int EPI>
__device__ __forceinline__ void epi_single(const GemmArgs& a, int m, int n, float v) {
  if constexpr (EPI == EPI_STORE) {
    ((T*)a.out)[(size_t)m * a.ldo + n] = from_f<T>(v);
  } else if constexpr (EPI == EPI_STORE_F32) {
    ((float*)a.out)[(size_t)m * a.ldo + n] = v;
  } else {  // EPI_RESID (out may alias resid: each element is read and written by one thread)
    const float r = to_f(((const T*)a.resid)[(size_t)m * a.ldr + n]);
    ((T*)a.out)[(size_t)m * a.ldo + n] = from_f<T>(r + v);
  }
}

// Paired epilogues: each 16-column block holds 8 a-columns followed by their 8 partners
// (weights repacked that way); c is the a-column, va/vb the pair.
template <typename T, int EPI>
__device__ __forceinline__ void epi_pair(const GemmArgs& a, int m, int c, float va, float vb) {
  if constexpr (EPI == EPI_SWIGLU) {
    const int f = (c >> 4) * 8 + (c & 7);
    const float s = va / (1.0f + __expf(-va));
    const size_t o = a.ostride > 0 ? frag_off(m, f, a.ostride) : (size_t)m * a.ldo + f;
    ((T*)a.out)[o] = from_f<T>(s * vb);
  } else {  // EPI_QKV
    const int D = a.d_model, hd = a.head_dim, half = hd >> 1;
    const int region = c / D, cr = c - region * D;
    const int h = cr / hd, jj = cr - h * hd;
    const int dj = (jj >> 4) * 8 + (jj & 7);  // rotary pair (dj, dj + hd/2)
    const int slot = a.row_sp[2 * m], pos = a.row_sp[2 * m + 1];
    if (region == 2) {
      T* dst = (T*)a.ring_v + (((size_t)slot * a.n_heads + h) * a.max_pos + pos) * hd;
      dst[dj] = from_f<T>(va);
      dst[dj + half] = from_f<T>(vb);
    } else {
      const float cs = a.rope_cs[((size_t)pos * half + dj) * 2];
      const float sn = a.rope_cs[((size_t)pos * half + dj) * 2 + 1];
      const float ra = va * cs - vb * sn, rb = vb * cs + va * sn;
      T* dst = region == 0 ? (T*)a.out + (size_t)m * a.ldo + h * hd
                           : (T*)a.ring_k + (((size_t)slot * a.n_heads + h) * a.max_pos + pos) * hd;
      dst[dj] = from_f<T>(ra);
      dst[dj + half] = from_f<T>(rb);
    }
  }
}

// Grouped epilogues (the bf16 GEMM, and the split-K reduction of both kernels): one call
// handles 8 consecutive output columns of a row with 16-byte (bf16) or 32-byte (fp32) accesses.
template <typename T>
__device__ __forceinline__ void load8(const T* p, T* r) {
  if constexpr (sizeof(T) == 2) {
    *(uint4*)r = *(const uint4*)p;
  } else {
    *(uint4*)r = *(const uint4*)p;
    *(uint4*)(r + 4) = *(const uint4*)(p + 4);
  }
}
template <typename T>
__device__ __forceinline__ void store8(T* p, const T* r) {
  if constexpr (sizeof(T) == 2) {
    *(uint4*)p = *(const uint4*)r;
  } else {
    *(uint4*)p = *(const uint4*)r;
    *(uint4*)(p + 4) = *(const uint4*)(r + 4);
  }
}

// Columns nc .. nc+7 (nc % 8 == 0) of row m.
template <typename T, int EPI>
__device__ __forceinline__ void epi_group8(const GemmArgs& a, int m, int nc, const float* v) {
  if constexpr (EPI == EPI_STORE_F32) {
    store8<float>((float*)a.out + (size_t)m * a.ldo + nc, v);
  } else {
    T r[8];
    if constexpr (EPI == EPI_RESID) {  // out may alias resid: each element is read, then written, by one thread
      T res[8];
      load8<T>((const T*)a.resid + (size_t)m * a.ldr + nc, res);
#pragma unroll
      for (int e = 0; e < 8; ++e) r[e] = from_f<T>(to_f(res[e]) + v[e]);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) r[e] = from_f<T>(v[e]);
    }
    store8<T>((T*)a.out + (size_t)m * a.ldo + nc, r);
  }
}

// The 16-column group starting at c (c % 16 == 0): a-columns c .. c+7, partners c+8 .. c+15.
template <typename T, int EPI>
__device__ __forceinline__ void epi_group16(const GemmArgs& a, int m, int c, const float* va, const float* vb) {
  T r0[8], r1[8];
  if constexpr (EPI == EPI_SWIGLU) {
    const int f = (c >> 4) * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) r0[e] = from_f<T>(va[e] / (1.0f + __expf(-va[e])) * vb[e]);
    store8<T>((T*)a.out + (a.ostride > 0 ? frag_off(m, f, a.ostride) : (size_t)m * a.ldo + f), r0);
  } else {  // EPI_QKV: rotary pairs (dj + e, dj + e + hd/2), e < 8
    const int D = a.d_model, hd = a.head_dim, half = hd >> 1;
    const int region = c / D, cr = c - region * D;
    const int h = cr / hd, dj = ((cr - h * hd) >> 4) * 8;
    const int slot = a.row_sp[2 * m], pos = a.row_sp[2 * m + 1];
    T* dst;
    if (region == 2) {
      dst = (T*)a.ring_v + (((size_t)slot * a.n_heads + h) * a.max_pos + pos) * hd;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        r0[e] = from_f<T>(va[e]);
        r1[e] = from_f<T>(vb[e]);
      }
    } else {
      float cs[16];
      load8<float>(a.rope_cs + ((size_t)pos * half + dj) * 2, cs);
      load8<float>(a.rope_cs + ((size_t)pos * half + dj) * 2 + 8, cs + 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        r0[e] = from_f<T>(va[e] * cs[2 * e] - vb[e] * cs[2 * e + 1]);
        r1[e] = from_f<T>(vb[e] * cs[2 * e] + va[e] * cs[2 * e + 1]);
      }
      dst = region == 0 ? (T*)a.out + (size_t)m * a.ldo + h * hd
                        : (T*)a.ring_k + (((size_t)slot * a.n_heads + h) * a.max_pos + pos) * hd;
    }
    store8<T>(dst + dj, r0);
    store8<T>(dst + dj + half, r1);
  }
}

// Tile configuration: BM rows (all packed rows for M <= 288) x four waves of WTN columns;
// PF weight k steps in flight per wave; DA activation stages in flight; OCC workgroups per CU.
template <int BM_, int WTN_, int PF_, int DA_, int OCC_>
struct GemmCfg {
  static constexpr int BM = BM_, WTN = WTN_, PF = PF_, DA = DA_, OCC = OCC_;
};

template <typename T, typename C, int EPI>
__global__ __launch_bounds__(256, C::OCC) void gemm_kernel(GemmArgs a) {
  constexpr int BM = C::BM, WTN = C::WTN, PF = C::PF, DA = C::DA;
  constexpr int BN = 4 * WTN;                  // four waves side by side along N
  constexpr int FM = BM / 16, NFB = WTN / 16;  // 16x16 blocks per wave
  constexpr int KPS = sizeof(T) == 2 ? 2 : 1;  // 32-wide k steps per 128-byte stage
  constexpr int VEC = 16 / (int)sizeof(T);     // elements per 16-byte chunk
  constexpr int A_IT = BM * 8 / 256;           // 16-byte activation chunks per thread per stage
  constexpr int UNR = PF / KPS;                // stages per unrolled block
  static_assert(BM % 32 == 0 && WTN % 16 == 0 && UNR % 2 == 0 && UNR % DA == 0 && A_IT >= 1, "tile shape");
    typedef typename Mma<T>::frag frag;

  __shared__ __attribute__((aligned(16))) T As[2][FM * KPS * 64 * 8];

  // Kp is a multiple of 32 * PF and every split is a whole number of PF k steps, so each
  // unrolled block of UNR stages is complete and the loop body has no guards.  Loads that
  // run past the split read clamped, valid addresses and are never consumed.
  const int n_mt = (a.M + BM - 1) / BM, n_nt = (a.N + BN - 1) / BN, S = a.splits;
  const int t = xcd_remap(blockIdx.x, n_mt * n_nt * S);
  const int mt = t % n_mt, rest = t / n_mt;
  const int sp = rest % S, nt = rest / S;
  const int m0 = mt * BM, n0 = nt * BN;
  const int ksteps = a.Kp >> 5;
  const int per = ((ksteps + S - 1) / S + PF - 1) / PF * PF;
  const int kb = min(ksteps, sp * per), ke = min(ksteps, kb + per);
  const int n_st = (ke - kb) / KPS;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int nb0 = (n0 + wave * WTN) >> 4;  // first 16-column block of this wave
  const int n_blocks = a.N >> 4;
  const T* __restrict__ A = (const T*)a.A;
  const T* __restrict__ Bf = (const T*)a.B;

  const T* brow[NFB];  // this lane's fragment stream of each of its column blocks
  static_for<0, NFB>([&](auto n) {
    brow[n] = Bf + (size_t)min(nb0 + (int)n, n_blocks - 1) * a.bstride + lane * 8;
  });
  frag bq[PF][NFB];
  auto load_b = [&](auto slot, int ks) {
    const size_t kc = (size_t)min(ks, ksteps - 1) * 512;
    static_for<0, NFB>([&](auto n) { bq[slot][n] = *(const frag*)(brow[n] + kc); });
  };

  // Activation chunks of this thread: row r, 16-byte column kl of each 128-byte stage.  Loads
  // are unconditional from clamped addresses: rows >= M only feed output rows that are never
  // stored, and k >= K meets zero weights (the packed weights are zero-padded to Kp), so the
  // clamped values, finite activations, contribute nothing.
  const T* arow[A_IT];
  int a_kl[A_IT], lds_off[A_IT];
  static_for<0, A_IT>([&](auto it) {
    const int ci = tid + it * 256;
    const int r = ci >> 3, kl = (ci & 7) * VEC;
    arow[it] = A + (size_t)min(m0 + r, a.M - 1) * a.lda;
    a_kl[it] = kl;
    lds_off[it] = ((((r >> 4) * KPS + (kl >> 5)) * 64) + (r & 15) + 16 * ((kl & 31) >> 3)) * 8 + (kl & 7);
  });
  u32x4 ra[DA][A_IT];
  auto load_a = [&](auto slot, int st) {
    const int k0 = (kb + st * KPS) * 32;
    static_for<0, A_IT>([&](auto it) { ra[slot][it] = *(const u32x4*)(arow[it] + min(k0 + a_kl[it], a.K - VEC)); });
  };
  auto store_a = [&](auto slot, auto buf) {
    static_for<0, A_IT>([&](auto it) { *(u32x4*)(&As[buf][lds_off[it]]) = ra[slot][it]; });
  };

  f32x4 acc[FM][NFB];
  static_for<0, FM>([&](auto i) { static_for<0, NFB>([&](auto n) { acc[i][n] = f32x4{0.f, 0.f, 0.f, 0.f}; }); });

  if (n_st > 0) {
    load_a(std::integral_constant<int, 0>{}, 0);
    static_for<0, PF>([&](auto p) { load_b(p, kb + p); });
    static_for<1, DA>([&](auto u) { load_a(u, u); });
    store_a(std::integral_constant<int, 0>{}, std::integral_constant<int, 0>{});
  }
  __syncthreads();

  for (int st0 = 0; st0 < n_st; st0 += UNR) {
    static_for<0, UNR>([&](auto u) {
      constexpr int U = decltype(u)::value;
      const int st = st0 + U;
      constexpr int buf = U & 1;  // st0 is a multiple of UNR (even), so buffers and slots are static
      static_for<0, KPS>([&](auto j) {
        constexpr int slot = U * KPS + decltype(j)::value;
        static_for<0, FM>([&](auto i) {
          const frag af = *(const frag*)(&As[buf][((i * KPS + j) * 64 + lane) * 8]);
          static_for<0, NFB>([&](auto n) { acc[i][n] = Mma<T>::mma(af, bq[slot][n], acc[i][n]); });
        });
        load_b(std::integral_constant<int, slot>{}, kb + st * KPS + decltype(j)::value + PF);  // refill
      });
      store_a(std::integral_constant<int, (U + 1) % DA>{}, std::integral_constant<int, buf ^ 1>{});  // stage st+1
      load_a(std::integral_constant<int, U % DA>{}, st + DA);  // the slot stage st used
      __syncthreads();
    });
  }

  // ---------------- epilogue: lane holds rows m0+16i+4lg+e of column (nb0+n)*16+lr
  const int lr = lane & 15, lg = lane >> 4;
  static_for<0, FM>([&](auto i) {
    static_for<0, 4>([&](auto e) {
      const int m = m0 + i * 16 + lg * 4 + e;
      const bool row_ok = m < a.M;
      static_for<0, NFB>([&](auto n) {
        const int c = (nb0 + n) * 16 + lr;
        const float v = acc[i][n][decltype(e)::value];
        if constexpr (EPI == EPI_SWIGLU || EPI == EPI_QKV) {
          const float partner = __shfl_xor(v, 8);  // all lanes take part
          if (S == 1 && row_ok && c < a.N && (lr & 8) == 0) epi_pair<T, EPI>(a, m, c, v, partner);
        } else {
          if (S == 1 && row_ok && c < a.N) epi_single<T, EPI>(a, m, c, v);
        }
        if (S > 1 && row_ok && c < a.N) a.partial[((size_t)sp * a.M + m) * a.N + c] = v;
      });
    });
  });
}

// Sums the split-K partials in split order and applies the epilogue; one thread per 8 output
// columns of a row (per 16-column pair group for the paired epilogues).
template <typename T, int EPI>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(GemmArgs a) {
  constexpr bool paired = EPI == EPI_SWIGLU || EPI == EPI_QKV;
  constexpr int W = paired ? 16 : 8;  // columns per thread
  const int per_row = a.N / W;
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= (size_t)a.M * per_row) return;
  const int m = (int)(idx / per_row), c = (int)(idx % per_row) * W;
  const size_t plane = (size_t)a.M * a.N;
  float v[W];
#pragma unroll
  for (int e = 0; e < W; ++e) v[e] = 0.f;
  for (int sp = 0; sp < a.splits; ++sp) {
    float t[W];
    const float* src = a.partial + sp * plane + (size_t)m * a.N + c;
    load8<float>(src, t);
    if constexpr (paired) load8<float>(src + 8, t + 8);
#pragma unroll
    for (int e = 0; e < W; ++e) v[e] += t[e];
  }
  if constexpr (paired)
    epi_group16<T, EPI>(a, m, c, v, v + 8);
  else
    epi_group8<T, EPI>(a, m, c, v);
}

template <typename T, typename C>
static hipError_t gemm_launch_cfg(int epi, const GemmArgs& a, hipStream_t s) {
  const int tiles = ((a.M + C::BM - 1) / C::BM) * ((a.N + 4 * C::WTN - 1) / (4 * C::WTN)) * a.splits;
  dim3 grid(tiles), block(256);
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL((gemm_kernel<T, C, EPI_STORE>), grid, block, 0, s, a); break;
    case EPI_STORE_F32: hipLaunchKernelGGL((gemm_kernel<T, C, EPI_STORE_F32>), grid, block, 0, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL((gemm_kernel<T, C, EPI_RESID>), grid, block, 0, s, a); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm_kernel<T, C, EPI_SWIGLU>), grid, block, 0, s, a); break;
    case EPI_QKV: hipLaunchKernelGGL((gemm_kernel<T, C, EPI_QKV>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <typename T>
static hipError_t reduce_launch(int epi, const GemmArgs& a, hipStream_t s) {
  const bool paired = epi == EPI_SWIGLU || epi == EPI_QKV;
  if (a.N % 16) return hipErrorInvalidValue;
  const size_t n = (size_t)a.M * (a.N / (paired ? 16 : 8));
  dim3 grid((unsigned)((n + 255) / 256)), block(256);
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL((splitk_reduce_kernel<T, EPI_STORE>), grid, block, 0, s, a); break;
    case EPI_STORE_F32: hipLaunchKernelGGL((splitk_reduce_kernel<T, EPI_STORE_F32>), grid, block, 0, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL((splitk_reduce_kernel<T, EPI_RESID>), grid, block, 0, s, a); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((splitk_reduce_kernel<T, EPI_SWIGLU>), grid, block, 0, s, a); break;
    case EPI_QKV: hipLaunchKernelGGL((splitk_reduce_kernel<T, EPI_QKV>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// fp32 tiles (small models): BM rows x four waves of 32 columns, two workgroups per CU; weight
// fragments stream through a per-wave register ring 4 k steps deep, activations through a
// 4-deep register ring into double-buffered LDS.
typedef GemmCfg<32, 32, 4, 4, 2> CfgF32S;
typedef GemmCfg<96, 32, 4, 4, 2> CfgF32M;
typedef GemmCfg<128, 32, 4, 4, 2> CfgF32L;

// 32 rows for decode-sized steps, else whichever of 96 and 128 pads M the least.
static int bm_for_f32(int M) {
  if (M <= 32) return 32;
  return ((M + 95) / 96) * 96 < ((M + 127) / 128) * 128 ? 96 : 128;
}

static hipError_t gemm_dispatch_f32(int epi, const GemmArgs& a, hipStream_t s) {
  const int bm = bm_for_f32(a.M);
  hipError_t e = bm == 32 ? gemm_launch_cfg<float, CfgF32S>(epi, a, s)
                 : bm == 96 ? gemm_launch_cfg<float, CfgF32M>(epi, a, s) : gemm_launch_cfg<float, CfgF32L>(epi, a, s);
  if (e != hipSuccess || a.splits <= 1 || a.partials_only) return e;
  return reduce_launch<float>(epi, a, s);
}

// ------------------------------------------------------------------ bf16 GEMM (32x32x16 MFMA)
// A workgroup is four waves side by side along N (32 columns each: a 128-column tile) over FM
// 32-row blocks (all packed rows up to 32 * FM) and one K split.  K advances in stages of
// four 16-wide k steps.
//  - Activations: a stage is FM x 4 fragment blocks of 1 KB, copied L2 -> LDS by
//    global_load_lds (each wave issues FM of them), with NBUF = 4 stages in flight; every wave
//    reads all of them from LDS, so each activation byte crosses L2 -> CU once per tile.
//  - Weights: each wave streams its own 32-column block into an 8-slot register ring two
//    stages ahead.  These loads are written as inline asm: the compiler would otherwise sink
//    them next to their use or drain them with waits of its own; the one vmcnt wait per stage
//    (issued with the barrier) covers them, and the ring's slots are fixed per unrolled stage.
//  - Per stage a wave waits and meets the barrier, issues the DMAs of stage st + 3, then runs
//    4 k steps of FM MFMAs with the next step's LDS reads issued ahead, refilling one weight
//    slot per step.
// Splits cover whole units of 4 stages (K is padded to a multiple of 256).
template <int FM, int NW, int EPI>
__global__ __launch_bounds__(64 * NW, 1) void gemm32_kernel(GemmArgs a) {
  constexpr int KS = 4, NBUF = 4, PFB = 8, BLK = 512;
  constexpr int SB = FM * KS;  // fragment blocks per stage
  constexpr int D = SB / NW;   // DMAs per wave per stage
  constexpr int P = PFB / KS;  // stages of weight lookahead
  static_assert(SB % NW == 0 && (NBUF * KS) % PFB == 0 && P >= 1 && P <= NBUF - 1, "pipeline shape");
  __shared__ __attribute__((aligned(1024))) bf16 As[NBUF][SB * BLK];

  const int tid = threadIdx.x, lane = tid & 63, nw = tid >> 6;
  const int n_blocks = (a.N + 31) >> 5, n_nt = (n_blocks + NW - 1) / NW;
  const int m_blocks = (a.M + 31) >> 5, n_mt = (m_blocks + FM - 1) / FM;
  const int S = a.splits;
  const int t = xcd_remap(blockIdx.x, n_mt * n_nt * S);
  const int mt = t % n_mt, rest = t / n_mt;
  const int sp = rest % S, nt = rest / S;
  const int ks16 = a.Kp >> 4;
  const int units = ks16 / (KS * NBUF), per = (units + S - 1) / S;
  const int kb = min(units, sp * per) * (KS * NBUF), ke = min(units, sp * per + per) * (KS * NBUF);
  const int n_st = (ke - kb) / KS;  // a multiple of NBUF
  const int nb_raw = nt * NW + nw;
  const int nb = min(nb_raw, n_blocks - 1);  // a wave past N streams a valid block and stores nothing

  const bf16* __restrict__ Ab = (const bf16*)a.A;
  const bf16* bp = (const bf16*)a.B + (size_t)nb * a.bstride + lane * 8;
  bf16x8 rb[PFB];
  auto load_b = [&](auto slot, int st, int j) {
    const int k = min(kb + st * KS + j, ks16 - 1);
    const bf16* src = bp + (size_t)k * BLK;
    bf16x8 v;
    asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(v) : "v"(src) : "memory");
    rb[slot] = v;
  };
  // stage st's block q (m-block q / KS of the tile, k step q % KS) lands at As[buf][q * BLK]
  auto dma = [&](auto buf, int st) {
    static_for<0, D>([&](auto d) {
      const int q = nw + NW * decltype(d)::value, mb = q / KS, j = q % KS;
      const int k = min(kb + st * KS + j, ks16 - 1);
      const int blk = min(mt * FM + mb, m_blocks - 1);  // rows past M: a valid block, never stored
      const bf16* src = Ab + (size_t)blk * a.astride + (size_t)k * BLK + lane * 8;
      __builtin_amdgcn_global_load_lds((const void*)src, (__attribute__((address_space(3))) void*)&As[buf][q * BLK],
                                       16, 0, 0);
    });
  };

  f32x16 acc[FM];
  static_for<0, FM>([&](auto i) { acc[i] = f32x16{}; });
  static_for<0, NBUF - 1>([&](auto b) {
    dma(b, b);
    __builtin_amdgcn_sched_barrier(0);
  });
  static_for<0, P>([&](auto s) {
    static_for<0, KS>([&](auto j) { load_b(std::integral_constant<int, s * KS + j>{}, s, j); });
  });
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the loop's waits count from a full ring
  __builtin_amdgcn_sched_barrier(0);

  for (int st0 = 0; st0 < n_st; st0 += NBUF) {
    static_for<0, NBUF>([&](auto u) {
      constexpr int U = decltype(u)::value;
      const int st = st0 + U;
      // Stage st's weights (the last loads of stage st - P) and activations (DMA'd NBUF - 1
      // stages back, earlier still) must have landed, in every wave (the barrier also frees
      // buffer (st - 1) % NBUF for the next DMA).  Loads issued after stage st's last weight
      // load: P - 1 stages of D DMAs + KS weight loads.
      constexpr int WAIT = (P - 1) * (D + KS);
      asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(WAIT) : "memory");
      dma(std::integral_constant<int, (U + NBUF - 1) % NBUF>{}, st + NBUF - 1);
      __builtin_amdgcn_sched_barrier(0);
      bf16x8 af[2][FM];
      static_for<0, FM>([&](auto i) { af[0][i] = *(const bf16x8*)(&As[U][(i * KS) * BLK + lane * 8]); });
      static_for<0, KS>([&](auto j) {
        constexpr int J = decltype(j)::value;
        constexpr int slot = (U * KS + J) % PFB;
        if constexpr (J + 1 < KS) {
          static_for<0, FM>([&](auto i) {
            af[(J + 1) & 1][i] = *(const bf16x8*)(&As[U][(i * KS + J + 1) * BLK + lane * 8]);
          });
        }
        __builtin_amdgcn_sched_barrier(0);
        static_for<0, FM>([&](auto i) {
          acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[J & 1][i], rb[slot], acc[i], 0, 0, 0);
        });
        load_b(std::integral_constant<int, slot>{}, st + P, J);
        __builtin_amdgcn_sched_barrier(0);
      });
    });
  }
  // The ring's last (unused) loads land before any of its registers can be reused.
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
  for (int p = 0; p < PFB; ++p) asm volatile("" : "+v"(rb[p]));

  // ---------------- epilogue.  The fp32 tile goes through LDS (the stage buffers hold exactly
  // 32 FM x 128 floats), then every thread handles 8 consecutive columns of a row (a 16-column
  // pair group for the paired epilogues) with vector accesses.  acc[i][r] is tile row
  // 32 i + 8 (r / 4) + 4 (lane / 32) + r % 4, tile column 32 nw + lane % 32.
  constexpr int BN_ = 32 * NW;
  static_assert(32 * FM * BN_ * 4 <= (int)sizeof(As), "epilogue tile must fit the stage buffers");
  float* T_ = (float*)&As[0][0];
  __syncthreads();  // every wave's last DMA has landed (vmcnt(0) above) and its LDS reads are done
  static_for<0, FM>([&](auto i) {
    static_for<0, 16>([&](auto r) {
      constexpr int R = decltype(r)::value;
      const int row = (int)decltype(i)::value * 32 + 8 * (R / 4) + 4 * (lane >> 5) + (R % 4);
      T_[row * BN_ + nw * 32 + (lane & 31)] = acc[i][R];
    });
  });
  __syncthreads();
  constexpr bool paired = EPI == EPI_SWIGLU || EPI == EPI_QKV;
  constexpr int W = paired ? 16 : 8;        // columns per item
  constexpr int BN = 32 * NW;               // tile columns
  constexpr int ITEMS = 32 * FM * (BN / W);
  const int m0 = mt * FM * 32, n0 = nt * BN;
  for (int it = tid; it < ITEMS; it += 64 * NW) {
    const int row = it / (BN / W), col = (it % (BN / W)) * W;
    const int m = m0 + row, nc = n0 + col;
    if (m >= a.M || nc >= a.N) continue;  // N % 16 == 0: a group is wholly inside or outside
    float v[W];
#pragma unroll
    for (int e = 0; e < W; e += 4) *(f32x4*)&v[e] = *(const f32x4*)&T_[row * BN + col + e];
    if (S > 1) {
      float* dst = a.partial + ((size_t)sp * a.M + m) * a.N + nc;
#pragma unroll
      for (int e = 0; e < W; e += 4) *(f32x4*)(dst + e) = *(const f32x4*)&v[e];
    } else if constexpr (paired) {
      epi_group16<bf16, EPI>(a, m, nc, v, v + 8);
    } else {
      epi_group8<bf16, EPI>(a, m, nc, v);
    }
  }
}

// Two-column-block variant for FM >= 2: the four waves form 2 row groups x 2 column groups of
// 64 columns (two 32-column weight blocks), so every activation fragment read from LDS feeds
// two MFMAs and the LDS read traffic per flop halves.  Row group 0 takes the first
// ceil(FM / 2) m-blocks, group 1 the rest.  Weights run two stages ahead (deeper rings measured
// slower: more requests in flight only queue).  Waits and epilogue as in gemm32_kernel.
template <int FM, int EPI>
__global__ __launch_bounds__(256, 1) void gemm32x2_kernel(GemmArgs a) {
  constexpr int KS = 4, NBUF = 4, PFB = 8, BLK = 512;
  constexpr int SB = FM * KS;  // fragment blocks per stage
  constexpr int D = SB / 4;    // DMAs per wave per stage
  constexpr int P = PFB / KS;  // stages of weight lookahead
  constexpr int MB0 = (FM + 1) / 2, MB1 = FM / 2;
  static_assert(FM >= 2 && SB % 4 == 0 && (NBUF * KS) % PFB == 0 && P >= 1, "pipeline shape");
  __shared__ __attribute__((aligned(1024))) bf16 As[NBUF][SB * BLK];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, rg = wave >> 1, cg = wave & 1;
  const int n_blocks = (a.N + 31) >> 5, n_nt = (n_blocks + 3) / 4;
  const int m_blocks = (a.M + 31) >> 5, n_mt = (m_blocks + FM - 1) / FM;
  const int S = a.splits;
  const int t = xcd_remap(blockIdx.x, n_mt * n_nt * S);
  const int mt = t % n_mt, rest = t / n_mt;
  const int sp = rest % S, nt = rest / S;
  const int ks16 = a.Kp >> 4;
  const int units = ks16 / (KS * NBUF), per = (units + S - 1) / S;
  const int kb = min(units, sp * per) * (KS * NBUF), ke = min(units, sp * per + per) * (KS * NBUF);
  const int n_st = (ke - kb) / KS;  // a multiple of NBUF
  // this wave's two weight blocks (past N: a valid block whose columns are never stored)
  const bf16* bp0 = (const bf16*)a.B + (size_t)min(nt * 4 + cg * 2, n_blocks - 1) * a.bstride + lane * 8;
  const bf16* bp1 = (const bf16*)a.B + (size_t)min(nt * 4 + cg * 2 + 1, n_blocks - 1) * a.bstride + lane * 8;
  const bf16* __restrict__ Ab = (const bf16*)a.A;

  auto dma = [&](auto buf, int st) {
    static_for<0, D>([&](auto d) {
      const int q = wave + 4 * decltype(d)::value, mb = q / KS, j = q % KS;
      const int k = min(kb + st * KS + j, ks16 - 1);
      const int blk = min(mt * FM + mb, m_blocks - 1);  // rows past M: a valid block, never stored
      const bf16* src = Ab + (size_t)blk * a.astride + (size_t)k * BLK + lane * 8;
      __builtin_amdgcn_global_load_lds((const void*)src, (__attribute__((address_space(3))) void*)&As[buf][q * BLK],
                                       16, 0, 0);
    });
  };
  float* T_ = (float*)&As[0][0];
  static_assert(32 * FM * 128 * 4 <= (int)sizeof(As), "epilogue tile must fit the stage buffers");

  // The main loop for a row group of MB m-blocks starting at MOFF; ends with the group's
  // accumulators parked in LDS as the fp32 tile [32 FM][128].
  auto body = [&](auto mb_c, auto moff_c) {
    constexpr int MB = decltype(mb_c)::value, MOFF = decltype(moff_c)::value;
    bf16x8 rb[PFB][2];
    auto load_b = [&](auto slot, int st, int j) {
      const int k = min(kb + st * KS + j, ks16 - 1);
      const bf16* s0 = bp0 + (size_t)k * BLK;
      const bf16* s1 = bp1 + (size_t)k * BLK;
      bf16x8 v0, v1;
      asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(v0) : "v"(s0) : "memory");
      asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(v1) : "v"(s1) : "memory");
      rb[slot][0] = v0;
      rb[slot][1] = v1;
    };
    f32x16 acc[MB][2];
    static_for<0, MB>([&](auto i) {
      acc[i][0] = f32x16{};
      acc[i][1] = f32x16{};
    });
    static_for<0, NBUF - 1>([&](auto b) {
      dma(b, b);
      __builtin_amdgcn_sched_barrier(0);
    });
    static_for<0, P>([&](auto s) {
      static_for<0, KS>([&](auto j) { load_b(std::integral_constant<int, s * KS + j>{}, s, j); });
    });
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the loop's waits count from a full ring
    __builtin_amdgcn_sched_barrier(0);

    for (int st0 = 0; st0 < n_st; st0 += NBUF) {
      static_for<0, NBUF>([&](auto u) {
        constexpr int U = decltype(u)::value;
        const int st = st0 + U;
        // Stage st needs its weights (the last loads of stage st - P) and its activations (the
        // DMA at the top of stage st - NBUF + 1); loads complete in order, so the wait counts
        // what was issued after the later of the two.  Per stage: D DMAs, then 2 KS weight loads.
        constexpr int WAIT = P <= NBUF - 1 ? (P - 1) * (D + 2 * KS) : 2 * KS + (NBUF - 2) * (D + 2 * KS);
        static_assert(WAIT <= 63, "vmcnt range");
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(WAIT) : "memory");
        dma(std::integral_constant<int, (U + NBUF - 1) % NBUF>{}, st + NBUF - 1);
        __builtin_amdgcn_sched_barrier(0);
        bf16x8 af[2][MB];
        static_for<0, MB>([&](auto i) {
          af[0][i] = *(const bf16x8*)(&As[U][((MOFF + decltype(i)::value) * KS) * BLK + lane * 8]);
        });
        static_for<0, KS>([&](auto j) {
          constexpr int J = decltype(j)::value;
          constexpr int slot = (U * KS + J) % PFB;
          if constexpr (J + 1 < KS) {
            static_for<0, MB>([&](auto i) {
              af[(J + 1) & 1][i] =
                  *(const bf16x8*)(&As[U][((MOFF + decltype(i)::value) * KS + J + 1) * BLK + lane * 8]);
            });
          }
          __builtin_amdgcn_sched_barrier(0);
          static_for<0, MB>([&](auto i) {
            acc[i][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[J & 1][i], rb[slot][0], acc[i][0], 0, 0, 0);
            acc[i][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[J & 1][i], rb[slot][1], acc[i][1], 0, 0, 0);
          });
          load_b(std::integral_constant<int, slot>{}, st + P, J);
          __builtin_amdgcn_sched_barrier(0);
        });
      });
    }
    // The ring's last (unused) loads land before any of its registers can be reused.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
    for (int p = 0; p < PFB; ++p) {
      asm volatile("" : "+v"(rb[p][0]));
      asm volatile("" : "+v"(rb[p][1]));
    }
    __syncthreads();  // every wave's DMAs have landed and its LDS reads are done
    static_for<0, MB>([&](auto i) {
      static_for<0, 2>([&](auto n) {
        static_for<0, 16>([&](auto r) {
          constexpr int R = decltype(r)::value;
          const int row = (MOFF + (int)decltype(i)::value) * 32 + 8 * (R / 4) + 4 * (lane >> 5) + (R % 4);
          T_[row * 128 + cg * 64 + (int)decltype(n)::value * 32 + (lane & 31)] = acc[i][n][R];
        });
      });
    });
  };
  if (rg == 0)
    body(std::integral_constant<int, MB0>{}, std::integral_constant<int, 0>{});
  else
    body(std::integral_constant<int, MB1>{}, std::integral_constant<int, MB0>{});
  __syncthreads();

  // ---------------- epilogue over the fp32 tile (as in gemm32_kernel)
  constexpr bool paired = EPI == EPI_SWIGLU || EPI == EPI_QKV;
  constexpr int W = paired ? 16 : 8;
  constexpr int ITEMS = 32 * FM * (128 / W);
  const int m0 = mt * FM * 32, n0 = nt * 128;
  for (int it = tid; it < ITEMS; it += 256) {
    const int row = it / (128 / W), col = (it % (128 / W)) * W;
    const int m = m0 + row, nc = n0 + col;
    if (m >= a.M || nc >= a.N) continue;  // N % 16 == 0: a group is wholly inside or outside
    float v[W];
#pragma unroll
    for (int e = 0; e < W; e += 4) *(f32x4*)&v[e] = *(const f32x4*)&T_[row * 128 + col + e];
    if (S > 1) {
      float* dst = a.partial + ((size_t)sp * a.M + m) * a.N + nc;
#pragma unroll
      for (int e = 0; e < W; e += 4) *(f32x4*)(dst + e) = *(const f32x4*)&v[e];
    } else if constexpr (paired) {
      epi_group16<bf16, EPI>(a, m, nc, v, v + 8);
    } else {
      epi_group8<bf16, EPI>(a, m, nc, v);
    }
  }
}

// NW-wave variant for 161..320 rows: the tile is 160 rows x 32 NW columns, each wave owning one
// 32-column weight block over all five row blocks, so no weight fragment is loaded twice and
// two row tiles fill the GPU where 288 x 128 tiles leave part of it idle.  Activations go
// through the LDS ring by DMA (issued by some of the waves, see below; every wave waits for its
// own loads and then the barrier), the weights stream into per-wave register rings as in
// gemm32x2_kernel.
// With a K split the kernel writes fp32 partial sums and splitk_reduce_kernel applies the
// epilogue; unsplit it applies the epilogue itself.
template <int FM, int NW, int EPI>
__global__ __launch_bounds__(64 * NW, 1) void gemm32c_kernel(GemmArgs a) {
  constexpr int KS = 4, NBUF = 4, PFB = 8, BLK = 512;
  constexpr int SB = FM * KS;  // fragment blocks per stage
  // the activation DMAs: with six waves, waves 0 and 1 share SIMDs with waves 4 and 5, so the
  // two waves alone on theirs (2 and 3) issue all of them; with four, every wave a quarter
  constexpr int NDW = NW == 6 ? 2 : 4;  // waves issuing DMAs
  constexpr int DW0 = NW == 6 ? 2 : 0;  // the first of them
  constexpr int DW = SB / NDW;          // DMAs per stage of each
  constexpr int P = PFB / KS;  // stages of weight lookahead
  constexpr int TC = 32 * NW;  // tile columns
  static_assert((NW == 4 || NW == 6) && SB % NDW == 0 && (NBUF * KS) % PFB == 0 && P >= 1, "pipeline shape");
  constexpr int AS_BYTES = NBUF * SB * BLK * 2, T_BYTES = 32 * FM * TC * 4;
  __shared__ __attribute__((aligned(1024))) char smem[AS_BYTES > T_BYTES ? AS_BYTES : T_BYTES];
  bf16(*As)[SB * BLK] = (bf16(*)[SB * BLK])smem;
  float* T_ = (float*)smem;  // the fp32 tile [32 FM][TC] once the main loop is done

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_blocks = (a.N + 31) >> 5, n_nt = (n_blocks + NW - 1) / NW;
  const int m_blocks = (a.M + 31) >> 5, n_mt = (m_blocks + FM - 1) / FM;
  const int S = a.splits;
  const int t = xcd_remap(blockIdx.x, n_mt * n_nt * S);
  const int mt = t % n_mt, rest = t / n_mt;
  const int sp = rest % S, nt = rest / S;
  const int ks16 = a.Kp >> 4;
  const int units = ks16 / (KS * NBUF), per = (units + S - 1) / S;
  const int kb = min(units, sp * per) * (KS * NBUF), ke = min(units, sp * per + per) * (KS * NBUF);
  const int n_st = (ke - kb) / KS;  // a multiple of NBUF
  // this wave's weight block (past N: a valid block whose columns are never stored)
  const bf16* bp = (const bf16*)a.B + (size_t)min(nt * NW + wave, n_blocks - 1) * a.bstride + lane * 8;
  const bf16* __restrict__ Ab = (const bf16*)a.A;

  auto body = [&](auto d_c) {
    constexpr int D = decltype(d_c)::value;  // DMAs per stage issued by this wave
    auto dma = [&](auto buf, int st) {
      static_for<0, D>([&](auto d) {
        const int q = (wave - DW0) + NDW * decltype(d)::value, mb = q / KS, j = q % KS;
        const int k = min(kb + st * KS + j, ks16 - 1);
        const int blk = min(mt * FM + mb, m_blocks - 1);  // rows past M: a valid block, never stored
        const bf16* src = Ab + (size_t)blk * a.astride + (size_t)k * BLK + lane * 8;
        __builtin_amdgcn_global_load_lds((const void*)src,
                                         (__attribute__((address_space(3))) void*)&As[buf][q * BLK], 16, 0, 0);
      });
    };
    bf16x8 rb[PFB];
    auto load_b = [&](auto slot, int st, int j) {
      const int k = min(kb + st * KS + j, ks16 - 1);
      const bf16* src = bp + (size_t)k * BLK;
      bf16x8 v;
      asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(v) : "v"(src) : "memory");
      rb[slot] = v;
    };
    f32x16 acc[FM];
    static_for<0, FM>([&](auto i) { acc[i] = f32x16{}; });
    static_for<0, NBUF - 1>([&](auto b) {
      dma(b, b);
      __builtin_amdgcn_sched_barrier(0);
    });
    static_for<0, P>([&](auto s) {
      static_for<0, KS>([&](auto j) { load_b(std::integral_constant<int, s * KS + j>{}, s, j); });
    });
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the loop's waits count from a full ring
    __builtin_amdgcn_sched_barrier(0);
    for (int st0 = 0; st0 < n_st; st0 += NBUF) {
      static_for<0, NBUF>([&](auto u) {
        constexpr int U = decltype(u)::value;
        const int st = st0 + U;
        // stage st needs its weights (the last loads of stage st - P) and activations (the DMA
        // of stage st - NBUF + 1); loads complete in order.  Per stage: D DMAs, then KS loads.
        constexpr int WAIT = P <= NBUF - 1 ? (P - 1) * (D + KS) : KS + (NBUF - 2) * (D + KS);
        static_assert(WAIT <= 63, "vmcnt range");
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(WAIT) : "memory");
        dma(std::integral_constant<int, (U + NBUF - 1) % NBUF>{}, st + NBUF - 1);
        __builtin_amdgcn_sched_barrier(0);
        bf16x8 af[2][FM];
        static_for<0, FM>([&](auto i) {
          af[0][i] = *(const bf16x8*)(&As[U][(decltype(i)::value * KS) * BLK + lane * 8]);
        });
        static_for<0, KS>([&](auto j) {
          constexpr int J = decltype(j)::value;
          constexpr int slot = (U * KS + J) % PFB;
          if constexpr (J + 1 < KS) {
            static_for<0, FM>([&](auto i) {
              af[(J + 1) & 1][i] = *(const bf16x8*)(&As[U][(decltype(i)::value * KS + J + 1) * BLK + lane * 8]);
            });
          }
          __builtin_amdgcn_sched_barrier(0);
          static_for<0, FM>([&](auto i) {
            acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[J & 1][i], rb[slot], acc[i], 0, 0, 0);
          });
          load_b(std::integral_constant<int, slot>{}, st + P, J);
          __builtin_amdgcn_sched_barrier(0);
        });
      });
    }
    // the ring's last (unused) loads land before any of its registers can be reused
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
    for (int p = 0; p < PFB; ++p) asm volatile("" : "+v"(rb[p]));
    __syncthreads();  // every wave's DMAs have landed and its LDS reads are done
    static_for<0, FM>([&](auto i) {
      static_for<0, 16>([&](auto r) {
        constexpr int R = decltype(r)::value;
        const int row = (int)decltype(i)::value * 32 + 8 * (R / 4) + 4 * (lane >> 5) + (R % 4);
        T_[row * TC + wave * 32 + (lane & 31)] = acc[i][R];
      });
    });
  };
  if (wave >= DW0 && wave < DW0 + NDW)
    body(std::integral_constant<int, DW>{});
  else
    body(std::integral_constant<int, 0>{});
  __syncthreads();

  // ---------------- epilogue over the fp32 tile (as in gemm32_kernel)
  constexpr bool paired = EPI == EPI_SWIGLU || EPI == EPI_QKV;
  constexpr int W = paired ? 16 : 8;
  constexpr int ITEMS = 32 * FM * (TC / W);
  const int m0 = mt * FM * 32, n0 = nt * TC;
  for (int it = tid; it < ITEMS; it += 64 * NW) {
    const int row = it / (TC / W), col = (it % (TC / W)) * W;
    const int m = m0 + row, nc = n0 + col;
    if (m >= a.M || nc >= a.N) continue;  // N % 16 == 0: a group is wholly inside or outside
    float v[W];
#pragma unroll
    for (int e = 0; e < W; e += 4) *(f32x4*)&v[e] = *(const f32x4*)&T_[row * TC + col + e];
    if (S > 1) {
      float* dst = a.partial + ((size_t)sp * a.M + m) * a.N + nc;
#pragma unroll
      for (int e = 0; e < W; e += 4) *(f32x4*)(dst + e) = *(const f32x4*)&v[e];
    } else if constexpr (paired) {
      epi_group16<bf16, EPI>(a, m, nc, v, v + 8);
    } else {
      epi_group8<bf16, EPI>(a, m, nc, v);
    }
  }
}

// The 160-row tiles are taken at 161..320 rows in two cases:
//  * six waves (192 columns), unsplit or split two ways over K, when that fills 3/4 of the GPU
//    or more in one pass (a 7B-shape step's gate/up projection: 2 x 115 = 230 workgroups; QKV:
//    2 x 64 x 2 = 256);
//  * four waves (128 columns) for narrow projections (N <= 4096) split four ways over K (the
//    output and down projections: 2 x 32 x 4 = 256 workgroups), which write half the fp32
//    partial sums of the 8-way split the 288 x 128 tile needs to fill the GPU.
constexpr int C6_FM = 5, C6_NW = 6;
static int c6_narrow(int M, int N, int Kp) {
  const int mb = (M + 31) / 32, nb = (N + 31) / 32, units = Kp / 256;
  if (mb <= C6_FM || mb > 2 * C6_FM || nb > 128 || units < 4) return 0;
  const int S = 4, per = (units + S - 1) / S;
  return (units + per - 1) / per;
}
static bool use_c6(const GemmArgs& a) {
  const int mb = (a.M + 31) / 32, nb = (a.N + 31) / 32;
  const int wgs = ((mb + C6_FM - 1) / C6_FM) * ((nb + C6_NW - 1) / C6_NW) * a.splits;
  if (a.splits > 1 && a.splits == c6_narrow(a.M, a.N, a.Kp)) return true;
  return a.splits <= 2 && mb > C6_FM && mb <= 2 * C6_FM && wgs >= 192 && wgs <= 256;
}

static hipError_t gemm32c_launch(int epi, const GemmArgs& a, hipStream_t s) {
  const int mb = (a.M + 31) / 32, nb = (a.N + 31) / 32;
  if (a.splits > 1 && a.splits == c6_narrow(a.M, a.N, a.Kp)) {  // narrow: four-wave 160 x 128 tile
    const dim3 grid(((mb + C6_FM - 1) / C6_FM) * ((nb + 3) / 4) * a.splits);
    hipLaunchKernelGGL((gemm32c_kernel<C6_FM, 4, EPI_STORE>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
  }
  const dim3 grid(((mb + C6_FM - 1) / C6_FM) * ((nb + C6_NW - 1) / C6_NW) * a.splits), block(64 * C6_NW);
  if (a.splits > 1) {  // partial sums only: one instance serves every epilogue
    hipLaunchKernelGGL((gemm32c_kernel<C6_FM, C6_NW, EPI_STORE>), grid, block, 0, s, a);
    return hipGetLastError();
  }
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL((gemm32c_kernel<C6_FM, C6_NW, EPI_STORE>), grid, block, 0, s, a); break;
    case EPI_STORE_F32: hipLaunchKernelGGL((gemm32c_kernel<C6_FM, C6_NW, EPI_STORE_F32>), grid, block, 0, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL((gemm32c_kernel<C6_FM, C6_NW, EPI_RESID>), grid, block, 0, s, a); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm32c_kernel<C6_FM, C6_NW, EPI_SWIGLU>), grid, block, 0, s, a); break;
    case EPI_QKV: hipLaunchKernelGGL((gemm32c_kernel<C6_FM, C6_NW, EPI_QKV>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

// 32-row blocks per tile: the smallest tile that holds every row (up to 10 blocks, 320 rows;
// FM = 10 fills the 160 KB of LDS), else the tile of 9 or 10 blocks with the fewest tiles and
// then the least padding.  A row's accumulation order is the same in every tile shape.
static int fm_for(int M) {
  const int mb = (M + 31) / 32;
  for (int fm : {1, 3, 5, 7, 9, 10})
    if (mb <= fm) return fm;
  const int t9 = (mb + 8) / 9, t10 = (mb + 9) / 10;
  return t10 < t9 || (t10 == t9 && t10 * 10 < t9 * 9) ? 10 : 9;
}

template <int FM, bool X2>
static hipError_t gemm32_launch(int epi, const GemmArgs& a, hipStream_t s) {
  const int n_nt = ((a.N + 31) / 32 + 3) / 4, n_mt = ((a.M + 31) / 32 + FM - 1) / FM;
  dim3 grid(n_mt * n_nt * a.splits), block(256);
#define AF_GEMM32(E)                                                                 \
  if constexpr (X2) hipLaunchKernelGGL((gemm32x2_kernel<FM, E>), grid, block, 0, s, a); \
  else hipLaunchKernelGGL((gemm32_kernel<FM, 4, E>), grid, block, 0, s, a);
  switch (epi) {
    case EPI_STORE: AF_GEMM32(EPI_STORE) break;
    case EPI_STORE_F32: AF_GEMM32(EPI_STORE_F32) break;
    case EPI_RESID: AF_GEMM32(EPI_RESID) break;
    case EPI_SWIGLU: AF_GEMM32(EPI_SWIGLU) break;
    case EPI_QKV: AF_GEMM32(EPI_QKV) break;
    default: return hipErrorInvalidValue;
  }
#undef AF_GEMM32
  return hipGetLastError();
}

// Split-K factor for a given tile count: none when the tiles alone fill most of the 256 CUs,
// else the largest factor (<= 8) that keeps every workgroup in one round, with at least one
// unit (256 k) per split.
static int splits_for(int tiles, int units) {
  if (tiles >= 160) return 1;
  return std::max(1, std::min(std::min(8, 256 / tiles), units));
}

static hipError_t gemm_dispatch_bf16(int epi, const GemmArgs& a, hipStream_t s) {
  if (a.astride <= 0 || a.Kp % 256 != 0 || a.astride < (long)a.Kp * 32 || a.bstride < (long)a.Kp * 32)
    return hipErrorInvalidValue;
  hipError_t e;
  if (use_c6(a)) {
    e = gemm32c_launch(epi, a, s);
    if (e != hipSuccess || a.splits <= 1 || a.partials_only) return e;
    return reduce_launch<bf16>(epi, a, s);
  }
  switch (fm_for(a.M)) {
    case 1: e = gemm32_launch<1, false>(epi, a, s); break;
    case 3: e = gemm32_launch<3, true>(epi, a, s); break;
    case 5: e = gemm32_launch<5, true>(epi, a, s); break;
    case 7: e = gemm32_launch<7, true>(epi, a, s); break;
    case 9: e = gemm32_launch<9, true>(epi, a, s); break;
    default: e = gemm32_launch<10, true>(epi, a, s); break;
  }
  if (e != hipSuccess || a.splits <= 1 || a.partials_only) return e;
  return reduce_launch<bf16>(epi, a, s);
}

int gemm_splits(int dtype, int M, int N, int Kp) {
  if (dtype == AF_BF16) {
    if (const int S = c6_narrow(M, N, Kp)) return S;
    const int fm = fm_for(M);
    const int tiles = (((M + 31) / 32 + fm - 1) / fm) * (((N + 31) / 32 + 3) / 4);
    return splits_for(tiles, Kp / gemm_k_align());
  }
  const int bm = bm_for_f32(M);
  const int tiles = ((M + bm - 1) / bm) * ((N + 127) / 128);
  if (tiles >= 160) return 1;
  return std::max(1, std::min(std::min(4, 256 / tiles), Kp / gemm_k_align()));
}

int gemm_k_align() { return 256; }

hipError_t launch_gemm(int dtype, int epi, const GemmArgs& a, hipStream_t s) {
  if (a.M <= 0 || a.N <= 0) return hipSuccess;
  if (a.splits < 1 || (a.splits > 1 && !a.partial)) return hipErrorInvalidValue;
  return dtype == AF_BF16 ? gemm_dispatch_bf16(epi, a, s) : gemm_dispatch_f32(epi, a, s);
}

// ------------------------------------------------------------------ segment-aware attention
// One workgroup = one (query tile of <= 64 rows of one segment, head).  Four waves own 16
// query rows each.  Key/value tiles of 64 positions of the segment's ring slot are staged in
// LDS (keys row-major, values transposed).  Scores are computed transposed, S^T = K . Q^T, so
// each lane holds scores of one query and the probabilities feed the P.V MFMA as its B
// operand without a lane exchange; softmax is online in the exp2 domain with the running
// max reduced across the four lanes that share a query.
// Single-row segments (decode steps), two per workgroup and head, each on half of the waves:
// one query against its slot's keys 0 .. pos0.  The waves of a half take chunks of 32 keys in
// turn.  A chunk issues all of its loads first (one memory latency per chunk): two lanes per key
// for the score (half a key row each), and for the value sum VEC dims of one dim group (l % DG)
// over the keys of its key group (l / DG + KG t), so every access is a 16-byte load.  Scores are fp32 dot products of the
// stored vectors (bf16 pairs through v_dot2); the softmax is online in the exp2 domain; the
// waves' (max, sum, output) are merged through LDS.  Separate from the tiled kernel so each
// keeps its own register budget.
template <typename T>
__device__ __forceinline__ float dot_vec(const uint4& k, const uint4& q, float acc) {
  if constexpr (sizeof(T) == 2) {
    typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;
    const unsigned kk[4] = {k.x, k.y, k.z, k.w}, qq[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int i = 0; i < 4; ++i)
      acc = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, kk[i]), __builtin_bit_cast(bf16x2, qq[i]), acc,
                                            false);
    return acc;
  } else {
    const float* kf = (const float*)&k;
    const float* qf = (const float*)&q;
#pragma unroll
    for (int i = 0; i < 4; ++i) acc += kf[i] * qf[i];
    return acc;
  }
}

// ROWS (1 or 2) single-row segments per workgroup: tiles first .. first + ROWS - 1 (those that
// exist), each on ATTN_WAVES / ROWS waves.  Two per workgroup halve the workgroups a packed
// step's decode rows take next to its query tiles.  Either way a row is computed as ATTN_WAVES
// virtual waves (virtual wave v takes chunks v, v + ATTN_WAVES, ..; a wave of a pair runs two
// of them one after the other) merged in virtual-wave order, so the result does not depend on
// how many rows share the workgroup.
template <typename T, int HD, int ROWS>
__device__ __forceinline__ void attention_decode_rows(const AttnArgs& a, int first) {
  constexpr int VEC = Chunk<T>::N;  // elements per 16 bytes
  constexpr int DG = HD / VEC;      // 16-byte chunks per key row
  constexpr int KH2 = DG / 2;       // chunks per half row (two lanes per key for the scores)
  constexpr int KG = 64 / DG;       // value key groups (lane / DG)
  constexpr int KPL = 32 / KG;      // values: keys per lane per 32-key chunk
  static_assert(DG % 2 == 0 && DG <= 64 && 64 % DG == 0 && 32 % KG == 0, "head_dim");
  static_assert(ROWS == 1 || ROWS == 2, "rows per workgroup");
  constexpr int VW = ATTN_WAVES;         // virtual waves per row
  constexpr int NW = ATTN_WAVES / ROWS;  // waves per row
  __shared__ float wm[ROWS][VW], wl[ROWS][VW];
  __shared__ __attribute__((aligned(16))) float wo[ROWS][VW][HD];
  __shared__ __attribute__((aligned(16))) uint4 qs[ROWS][DG];
  const int tid = threadIdx.x, lane = tid & 63, wave0 = tid >> 6;
  const int sub = ROWS == 1 ? 0 : wave0 / NW, wave = ROWS == 1 ? wave0 : wave0 % NW;  // row, wave within it
  const bool live = ROWS == 1 || first + sub < a.n_tiles;  // an odd count leaves the last half idle
  const int seg_i = a.tiles[2 * (live ? first + sub : first)];
  const int h = blockIdx.y;
  const DevSeg sg = a.segs[seg_i];
  const int kv_len = live ? sg.pos0 + 1 : 0;
  const size_t slot_off = ((size_t)sg.slot * a.n_heads + h) * a.max_pos * HD;
  const T* __restrict__ Kg = (const T*)a.ring_k + slot_off;
  const T* __restrict__ Vg = (const T*)a.ring_v + slot_off;
  // the query, the same for every lane of the row's waves, is read from LDS (broadcast reads)
  const int htid = tid - sub * NW * 64;
  if (live && htid < DG) qs[sub][htid] = ((const uint4*)((const T*)a.q + (size_t)sg.q_start * a.ldq + h * HD))[htid];
  __syncthreads();

  const int half = lane & 1, kl = lane >> 1;   // scores: key kl of the chunk, half row `half`
  const int dg = lane % DG, kgrp = lane / DG;  // values: dims [VEC dg, +VEC) of keys kgrp + KG t
#pragma unroll
  for (int r = 0; r < VW / NW; ++r) {
    const int v = wave + r * NW;  // the virtual wave
    float m_run = -INFINITY, l_run = 0.f, o[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) o[e] = 0.f;
    for (int c = v; c * 32 < kv_len; c += VW) {
      // keys past kv_len read a clamped valid key and score -inf
      const int j = c * 32 + kl;
      const uint4* krow = (const uint4*)(Kg + (size_t)min(j, kv_len - 1) * HD) + half * KH2;
      uint4 kv[KH2], vv[KPL];
#pragma unroll
      for (int pc = 0; pc < KH2; ++pc) kv[pc] = krow[pc];
#pragma unroll
      for (int t = 0; t < KPL; ++t)
        vv[t] = *(const uint4*)(Vg + (size_t)min(c * 32 + kgrp + KG * t, kv_len - 1) * HD + dg * VEC);
      float dot = 0.f;
#pragma unroll
      for (int pc = 0; pc < KH2; ++pc) dot = dot_vec<T>(kv[pc], qs[sub][half * KH2 + pc], dot);
      dot += __shfl_xor(dot, 1);
      const float sc = j < kv_len ? dot * a.scale_log2 : -INFINITY;
      float cm = sc;
#pragma unroll
      for (int off = 32; off > 1; off >>= 1) cm = fmaxf(cm, __shfl_xor(cm, off));
      const float m_new = fmaxf(m_run, cm);
      const float p = exp2f(sc - m_new);
      float ps = half ? 0.f : p;  // each key is held by two lanes
#pragma unroll
      for (int off = 32; off > 0; off >>= 1) ps += __shfl_xor(ps, off);
      const float corr = exp2f(m_run - m_new);  // 0 on the first chunk (m_run = -inf)
      l_run = l_run * corr + ps;
      m_run = m_new;
#pragma unroll
      for (int e = 0; e < VEC; ++e) o[e] *= corr;
      // lane covers dims [VEC dg, +VEC) of keys c*32 + kgrp + KG t (masked keys carry p = 0)
#pragma unroll
      for (int t = 0; t < KPL; ++t) {
        const float pj = __shfl(p, 2 * (kgrp + KG * t));
        T vt[VEC];
        __builtin_memcpy(vt, &vv[t], 16);
#pragma unroll
        for (int e = 0; e < VEC; ++e) o[e] += pj * to_f(vt[e]);
      }
    }
    // ---- merge the key groups of the virtual wave; park its state for the row's merge
#pragma unroll
    for (int off = DG; off < 64; off <<= 1)
#pragma unroll
      for (int e = 0; e < VEC; ++e) o[e] += __shfl_xor(o[e], off);
    if (lane == 0) {
      wm[sub][v] = m_run;
      wl[sub][v] = l_run;
    }
    if (lane < DG)
#pragma unroll
      for (int e = 0; e < VEC; ++e) wo[sub][v][dg * VEC + e] = o[e];
  }
  __syncthreads();
  if (live && wave == 0 && lane < DG) {
    float M = wm[sub][0];
#pragma unroll
    for (int w = 1; w < VW; ++w) M = fmaxf(M, wm[sub][w]);
    float L = 0.f, acc[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) acc[e] = 0.f;
#pragma unroll
    for (int w = 0; w < VW; ++w) {
      const float f = wm[sub][w] == -INFINITY ? 0.f : exp2f(wm[sub][w] - M);  // a virtual wave with no chunk
      L += wl[sub][w] * f;
#pragma unroll
      for (int e = 0; e < VEC; ++e) acc[e] += wo[sub][w][dg * VEC + e] * f;
    }
    const float inv = 1.0f / L;
    T r[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) r[e] = from_f<T>(acc[e] * inv);
    const int k0 = h * HD + dg * VEC;
    T* dst = a.ostride > 0 ? (T*)a.o + frag_off(sg.q_start, k0, a.ostride) : (T*)a.o + (size_t)sg.q_start * a.ldo + k0;
    *(uint4*)dst = *(const uint4*)r;
  }
}

// Query tiles of multi-row segments.  The next key/value tile is loaded into registers while
// the current one is processed from LDS (one memory latency per segment, not per tile).
template <typename T, int HD>
__device__ __forceinline__ void attention_prefill_tile(const AttnArgs& a, int tile) {
  constexpr int VEC = Chunk<T>::N;
  constexpr int KROW = HD + VEC;            // padded key row (elements)
  constexpr int VROW = ATTN_BKV + VEC;      // padded transposed-value row
  constexpr int KST = HD / 32;              // MFMA k steps over the head dimension
  constexpr int DB = HD / 16;               // 16-dim output blocks
  constexpr int CPR = HD / VEC;             // 16-byte chunks per key row
  constexpr int NCH = ATTN_BKV * CPR / 256; // chunks of K (and of V) per thread per tile
  static_assert((ATTN_BKV * CPR) % 256 == 0, "tile shape");
  typedef typename Mma<T>::frag frag;

  // two key groups of four waves: group g takes key tiles g, g + 2, g + 4, .. of the segment
  // with buffers of its own; the groups' partial softmax states are merged at the end
  __shared__ __attribute__((aligned(16))) T Ks[2][ATTN_BKV * KROW];
  __shared__ __attribute__((aligned(16))) T Vt[2][HD * VROW];

  const int lane = threadIdx.x & 63, grp = threadIdx.x >> 8, wave = (threadIdx.x >> 6) & 3;
  const int tid = threadIdx.x & 255;  // position within the key group
  const int lr = lane & 15, lg = lane >> 4;
  const int seg_i = a.tiles[2 * tile], i0 = a.tiles[2 * tile + 1];
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
    const T* qrow = (const T*)a.q + (size_t)(sg.q_start + qi_c) * a.ldq + h * HD;
#pragma unroll
    for (int s = 0; s < KST; ++s) qf[s] = *(const frag*)(qrow + s * 32 + lg * 8);
  }

  f32x4 oacc[DB];
#pragma unroll
  for (int d = 0; d < DB; ++d) oacc[d] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run = -INFINITY, l_run = 0.f;

  // One tile's keys and values in registers.  Keys: thread t holds 16-byte chunk t % CPR of
  // keys t / CPR + KR j (row-major LDS writes, one key row per CPR lanes).  Values: thread t
  // holds KPT consecutive keys (t % KGV) * KPT .. of dim chunk t / KGV, so that after a
  // transpose in registers each dim's KPT keys go to LDS as one contiguous write.
  constexpr int KR = 256 / CPR;          // key rows per pass
  constexpr int KPT = NCH;               // values: keys per thread
  constexpr int KGV = ATTN_BKV / KPT;    // values: key groups
  static_assert(KGV * CPR == 256, "value mapping");
  uint4 kreg[NCH], vreg[NCH];
  const int kc = tid % CPR, kr = tid / CPR;
  const int vg = tid % KGV, vc = tid / KGV;
  auto load_tile = [&](int kb0) {
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      const int key = kb0 + kr + KR * j;
      kreg[j] = key < kv_end ? *(const uint4*)(Kg + (size_t)key * HD + kc * VEC) : zero4();
      const int vkey = kb0 + vg * KPT + j;
      vreg[j] = vkey < kv_end ? *(const uint4*)(Vg + (size_t)vkey * HD + vc * VEC) : zero4();
    }
  };
  const int n_kt = (kv_end + ATTN_BKV - 1) / ATTN_BKV;
  const int n_it = (n_kt + 1) / 2;  // both groups run the same iterations (and barriers)
  load_tile(grp * ATTN_BKV);        // keys past kv_end load as zeros
  for (int it = 0; it < n_it; ++it) {
    const int kt = 2 * it + grp;
    const int kb0 = kt * ATTN_BKV;
    // ---- park the tile in LDS: keys row-major, values transposed
    __syncthreads();  // the previous tile's LDS reads are done
#pragma unroll
    for (int j = 0; j < NCH; ++j) *(uint4*)(&Ks[grp][(kr + KR * j) * KROW + kc * VEC]) = kreg[j];
    {
      T vt[NCH][VEC];
#pragma unroll
      for (int j = 0; j < NCH; ++j) __builtin_memcpy(vt[j], &vreg[j], 16);
#pragma unroll
      for (int e = 0; e < VEC; ++e) {
        T col[KPT];
#pragma unroll
        for (int j = 0; j < KPT; ++j) col[j] = vt[j][e];
        T* dst = &Vt[grp][(vc * VEC + e) * VROW + vg * KPT];
        if constexpr (KPT * sizeof(T) == 4) {
          *(unsigned*)dst = *(const unsigned*)col;
        } else if constexpr (KPT * sizeof(T) == 8) {
          *(uint2*)dst = *(const uint2*)col;
        } else {
          static_assert((KPT * sizeof(T)) % 16 == 0, "value chunk");
#pragma unroll
          for (int q = 0; q < (int)(KPT * sizeof(T)) / 16; ++q) *(uint4*)(dst + q * 16 / sizeof(T)) = *(const uint4*)(col + q * 16 / sizeof(T));
        }
      }
    }
    __syncthreads();
    if (kt + 2 < n_kt) load_tile(kb0 + 2 * ATTN_BKV);  // this group's next tile, in flight meanwhile

    if (wave_rows > 0 && kb0 <= wave_last_pos) {
      // ---- S^T = K . Q^T for 4 blocks of 16 keys
      float p[4][4];
      float tmax = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) {
        f32x4 sacc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < KST; ++s) {
          const frag kf = *(const frag*)(&Ks[grp][(kb * 16 + lr) * KROW + s * 32 + lg * 8]);
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
      // a row may not have seen any key yet (key group 1's first tile can lie wholly past some
      // rows): then every score so far is -inf, and 0 stands in as the reference so that the
      // probabilities and the correction come out 0 instead of exp2(-inf - -inf)
      const float m_ref = m_new == -INFINITY ? 0.f : m_new;
      const float corr = exp2f(m_run - m_ref);  // m_run = -inf before the row's first key -> 0
      float psum = 0.f;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float pe = exp2f(p[kb][e] - m_ref);
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
          // keys lg * 4 .. +3 and 16 + lg * 4 .. +3 of the chunk: two aligned 4-element reads
          const T* vrow = &Vt[grp][(d * 16 + lr) * VROW + c * 32 + lg * 4];
          frag vf;
          if constexpr (sizeof(T) == 2) {
            typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4_;
            const bf16x4_ lo = *(const bf16x4_*)vrow, hi = *(const bf16x4_*)(vrow + 16);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              vf[e] = lo[e];
              vf[4 + e] = hi[e];
            }
          } else {
            const f32x4 lo = *(const f32x4*)vrow, hi = *(const f32x4*)(vrow + 16);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              vf[e] = lo[e];
              vf[4 + e] = hi[e];
            }
          }
          oacc[d] = Mma<T>::mma(vf, pf, oacc[d]);
          if constexpr (sizeof(T) == 2) oacc[d] = Mma<T>::mma(vf, pf_lo, oacc[d]);
        }
      }
    }
  }

  // ---- merge key group 1 into group 0 (per lane: the same query and output dims in both)
  constexpr int NF = 2 + 4 * DB;  // m, l, the output accumulators
  static_assert(4 * 64 * NF * sizeof(float) <= sizeof(Ks), "merge buffer");
  float* mb = (float*)&Ks[0][0] + (size_t)wave * NF * 64 + lane;
  __syncthreads();  // every wave is done with the key/value buffers
  if (grp == 1) {
    mb[0] = m_run;
    mb[64] = l_run;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int e = 0; e < 4; ++e) mb[(2 + 4 * d + e) * 64] = oacc[d][e];
  }
  __syncthreads();
  if (grp == 1) return;
  {
    const float m1 = mb[0], l1 = mb[64];
    const float M = fmaxf(m_run, m1);
    const float f0 = m_run == -INFINITY ? 0.f : exp2f(m_run - M), f1 = m1 == -INFINITY ? 0.f : exp2f(m1 - M);
    l_run = l_run * f0 + l1 * f1;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int e = 0; e < 4; ++e) oacc[d][e] = oacc[d][e] * f0 + mb[(2 + 4 * d + e) * 64] * f1;
  }
  if (wave_rows <= 0 || !q_ok) return;
  float l_tot = l_run + __shfl_xor(l_run, 16);
  l_tot += __shfl_xor(l_tot, 32);
  const float inv = 1.0f / l_tot;
  const int m = sg.q_start + qi;
  if (a.ostride > 0) {  // fragment-tiled for the output projection: 4 consecutive k are contiguous
#pragma unroll
    for (int d = 0; d < DB; ++d) {
      T* dst = (T*)a.o + frag_off(m, h * HD + d * 16 + lg * 4, a.ostride);
#pragma unroll
      for (int e = 0; e < 4; ++e) dst[e] = from_f<T>(oacc[d][e] * inv);
    }
  } else {
    T* orow = (T*)a.o + (size_t)m * a.ldo + h * HD;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int e = 0; e < 4; ++e) orow[d * 16 + lg * 4 + e] = from_f<T>(oacc[d][e] * inv);
  }
}

// One launch for the whole step: work tiles [0, n_multi) are query tiles of multi-row segments
// (ordered longest first, so they start first), the rest single-row segments.
// Blocks [0, n_multi) of the query-tile instance take the query tiles, its other blocks pairs of
// single-row tiles (n_multi + 2 (blockIdx.x - n_multi) and the next); the decode-only instance
// takes one single-row tile per block (n_multi + blockIdx.x), on all of its waves.
template <typename T, int HD, bool PREFILL>
__global__ __launch_bounds__(64 * ATTN_WAVES, !PREFILL ? 4 : 2) void attention_kernel(AttnArgs a) {
  const int b = blockIdx.x;
  if constexpr (PREFILL) {
    if (b < a.n_multi)
      attention_prefill_tile<T, HD>(a, b);
    else
      attention_decode_rows<T, HD, 2>(a, a.n_multi + 2 * (b - a.n_multi));
  } else {
    attention_decode_rows<T, HD, 1>(a, a.n_multi + b);
  }
}

// Query tiles and decode rows share one launch, query tiles first; the decode-only kernel has
// no query-tile LDS and registers and so fits more workgroups per CU, which pays once the decode
// rows alone would more than fill the GPU twice over (a second launch then costs less).
template <typename T, int HD>
static void attention_launch(const AttnArgs& a0, int n_tiles, hipStream_t s) {
  AttnArgs a = a0;
  a.n_tiles = n_tiles;
  const dim3 block(64 * ATTN_WAVES);
  const int n_single = n_tiles - a.n_multi, n_pairs = (n_single + 1) / 2;
  if (a.n_multi == 0) {
    hipLaunchKernelGGL((attention_kernel<T, HD, false>), dim3(n_tiles, a.n_heads), block, 0, s, a);
  } else if ((long)n_pairs * a.n_heads <= 256) {
    hipLaunchKernelGGL((attention_kernel<T, HD, true>), dim3(a.n_multi + n_pairs, a.n_heads), block, 0, s, a);
  } else {
    hipLaunchKernelGGL((attention_kernel<T, HD, true>), dim3(a.n_multi, a.n_heads), block, 0, s, a);
    if (n_single > 0)  // the decode-only instance: its blocks start at the first single-row tile
      hipLaunchKernelGGL((attention_kernel<T, HD, false>), dim3(n_single, a.n_heads), block, 0, s, a);
  }
}

// tiles[0, n_multi) are query tiles of multi-row segments, tiles[n_multi, n_tiles) the
// single-row segments.
hipError_t launch_attention(int dtype, int head_dim, const AttnArgs& a, int n_tiles, hipStream_t s) {
  if (n_tiles <= 0) return hipSuccess;
  if (a.n_multi < 0 || a.n_multi > n_tiles || (head_dim != 64 && head_dim != 128)) return hipErrorInvalidValue;
  if (dtype == AF_BF16) {
    if (head_dim == 128) attention_launch<bf16, 128>(a, n_tiles, s);
    else attention_launch<bf16, 64>(a, n_tiles, s);
  } else {
    if (head_dim == 128) attention_launch<float, 128>(a, n_tiles, s);
    else attention_launch<float, 64>(a, n_tiles, s);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------ RMSNorm
// One workgroup of NORM_THREADS threads per output row (a 4096-wide bf16 row is one 16-byte
// chunk per thread: one memory latency); rows[] optionally selects the input row.  The
// output is row-major (row stride ldy) or, with ystride > 0, fragment-tiled for the GEMM that
// consumes it.  bf16 rows with D % 8 == 0 move 16 bytes per thread access.
constexpr int NORM_THREADS = 512;

// Sum over the workgroup of one value per thread, in a fixed order (lanes by xor shuffles, then
// the waves in order); the same order in every kernel that normalises a row.
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
  if (vec) {
    for (int i = threadIdx.x * V; i < D; i += NORM_THREADS * V) {
      T v[V];
      *(uint4*)v = *(const uint4*)(xr + i);
#pragma unroll
      for (int e = 0; e < V; ++e) ss += to_f(v[e]) * to_f(v[e]);
    }
  } else {
    for (int i = threadIdx.x; i < D; i += NORM_THREADS) {
      const float v = to_f(xr[i]);
      ss += v * v;
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

hipError_t launch_rmsnorm(int dtype, const void* x, int ldx, const int32_t* rows, const void* g, void* y, int ldy,
                          long ystride, int n_rows, int D, float eps, hipStream_t s) {
  if (n_rows <= 0) return hipSuccess;
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
      for (int e = 0; e < 8; ++e) ss += to_f(r[e]) * to_f(r[e]);
    }
  } else {
    for (int i = threadIdx.x; i < D; i += NORM_THREADS) {
      float v = 0.f;
      for (int sp = 0; sp < splits; ++sp) v += partial[sp * plane + (size_t)m * D + i];
      const T r = from_f<T>(to_f(xr[i]) + v);
      xr[i] = r;
      ss += to_f(r) * to_f(r);
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
