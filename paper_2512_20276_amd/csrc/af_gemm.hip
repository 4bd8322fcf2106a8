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
#include "af_device.h"

namespace af {

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
  n += a.col0;
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
  c += a.col0;
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
      const float ra = fmaf(va, cs, -(vb * sn)), rb = fmaf(vb, cs, va * sn);  // as epi_group16
      T* dst = region == 0 ? (T*)a.out + (size_t)m * a.ldo + h * hd
                           : (T*)a.ring_k + (((size_t)slot * a.n_heads + h) * a.max_pos + pos) * hd;
      dst[dj] = from_f<T>(ra);
      dst[dj + half] = from_f<T>(rb);
    }
  }
}

// Columns nc .. nc+7 (nc % 8 == 0) of row m.
template <typename T, int EPI>
__device__ __forceinline__ void epi_group8(const GemmArgs& a, int m, int nc, const float* v) {
  nc += a.col0;
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

// What the QKV epilogue needs besides the sums for one 16-column group of row m: the region
// (queries, keys, values), head, rotary offset, the row's ring slot and position, and the
// rotary (cos, sin) pairs; loaded ahead of the sums where the sums come from memory.
struct QkvRow {
  int region, h, dj, slot, pos;
  float cs[16];
  __device__ __forceinline__ void load(const GemmArgs& a, int m, int c) {
    const int D = a.d_model, hd = a.head_dim, half = hd >> 1;
    c += a.col0;
    region = c / D;
    const int cr = c - region * D;
    h = cr / hd;
    dj = ((cr - h * hd) >> 4) * 8;
    slot = a.row_sp[2 * m];
    pos = a.row_sp[2 * m + 1];
    if (region != 2) {
      load8<float>(a.rope_cs + ((size_t)pos * half + dj) * 2, cs);
      load8<float>(a.rope_cs + ((size_t)pos * half + dj) * 2 + 8, cs + 8);
    }
  }
};

// The 16-column group starting at c (c % 16 == 0): a-columns c .. c+7, partners c+8 .. c+15.
template <typename T, int EPI>
__device__ __forceinline__ void epi_group16(const GemmArgs& a, int m, int c, const float* va, const float* vb,
                                            const QkvRow* pre = nullptr) {
  T r0[8], r1[8];
  if constexpr (EPI == EPI_SWIGLU) {
    const int f = ((c + a.col0) >> 4) * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) r0[e] = from_f<T>(va[e] / (1.0f + __expf(-va[e])) * vb[e]);
    store8<T>((T*)a.out + (a.ostride > 0 ? frag_off(m, f, a.ostride) : (size_t)m * a.ldo + f), r0);
  } else {  // EPI_QKV: rotary pairs (dj + e, dj + e + hd/2), e < 8
    QkvRow q;
    if (pre) q = *pre;
    else q.load(a, m, c);
    const int hd = a.head_dim, half = hd >> 1;
    T* dst;
    if (q.region == 2) {
      dst = (T*)a.ring_v + (((size_t)q.slot * a.n_heads + q.h) * a.max_pos + q.pos) * hd;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        r0[e] = from_f<T>(va[e]);
        r1[e] = from_f<T>(vb[e]);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        // explicit fused multiply-adds: every kernel that applies this epilogue rounds alike
        r0[e] = from_f<T>(fmaf(va[e], q.cs[2 * e], -(vb[e] * q.cs[2 * e + 1])));
        r1[e] = from_f<T>(fmaf(vb[e], q.cs[2 * e], va[e] * q.cs[2 * e + 1]));
      }
      dst = q.region == 0 ? (T*)a.out + (size_t)m * a.ldo + q.h * hd
                          : (T*)a.ring_k + (((size_t)q.slot * a.n_heads + q.h) * a.max_pos + q.pos) * hd;
    }
    store8<T>(dst + q.dj, r0);
    store8<T>(dst + q.dj + half, r1);
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
  // every load is issued before any sum waits on one: the epilogue's row data, then all the
  // partial sums (up to MAXS splits at once); they are added in split order
  QkvRow q;
  if constexpr (EPI == EPI_QKV) q.load(a, m, c);
  constexpr int MAXS = 4;
  float t[MAXS][W];
#pragma unroll
  for (int sp = 0; sp < MAXS; ++sp)
    if (sp < a.splits) {
      const float* src = a.partial + sp * plane + (size_t)m * a.N + c;
      load8<float>(src, t[sp]);
      if constexpr (paired) load8<float>(src + 8, t[sp] + 8);
    }
  float v[W];
#pragma unroll
  for (int e = 0; e < W; ++e) v[e] = 0.f;
#pragma unroll
  for (int sp = 0; sp < MAXS; ++sp)
    if (sp < a.splits)
#pragma unroll
      for (int e = 0; e < W; ++e) v[e] += t[sp][e];
  for (int sp = MAXS; sp < a.splits; ++sp) {
    float u[W];
    const float* src = a.partial + sp * plane + (size_t)m * a.N + c;
    load8<float>(src, u);
    if constexpr (paired) load8<float>(src + 8, u + 8);
#pragma unroll
    for (int e = 0; e < W; ++e) v[e] += u[e];
  }
  if constexpr (paired)
    epi_group16<T, EPI>(a, m, c, v, v + 8, EPI == EPI_QKV ? &q : nullptr);
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

// Wide tile for many rows: 32 FM rows x 32 CB NW columns on NW waves, each owning CB 32-column
// weight blocks over all FM row blocks (as gemm32c_kernel does for 160 rows), so no weight
// fragment is loaded twice.  Per byte loaded into the CU the 288 x 256 tile does 1.5x the MFMA
// work of the 288 x 128 one (288 + 256 bytes per row of K for 288 x 256 outputs, against
// 288 + 128 for 288 x 128).  Every activation fragment read from LDS feeds CB MFMAs: with
// eight waves of one block each (two waves per SIMD, 144 accumulator registers) the LDS reads
// of a 16-k step (72 KB) take as long as its MFMAs; with four waves of two blocks (one wave per
// SIMD, 288 accumulator registers) they take half, and each wave double-buffers its
// fragments, as no other wave on its SIMD covers the LDS latency.  The weights run two k steps
// ahead.  Activations by DMA from waves 0..3; the fp32 tile goes through the LDS ring three
// row blocks per pass.  (Three row groups of four column groups, each wave two weight blocks,
// measured no faster: each weight fragment was then requested once per row group.  Four
// waves of two blocks, 256 x 256 with 256 accumulator registers, measured 1.2x slower for
// gate/up at 2264 rows: one wave per SIMD leaves every wait of a wave on the matrix core.)
template <int FM, int NW, int CB, int EPI>
__global__ __launch_bounds__(64 * NW, 1) void gemm32w_kernel(GemmArgs a) {
  constexpr int KS = 4, NBUF = 4, PFB = 2, BLK = 512, TN = 32 * CB * NW, PB = 3;
  constexpr int AFB = NW <= 4 ? 2 : 1;  // activation fragment buffers per wave
  constexpr int SB = FM * KS;           // fragment blocks per stage
  constexpr int DW = SB / 4;            // DMAs per stage of each of waves 0..3
  constexpr int NPASS = (FM + PB - 1) / PB;
  static_assert(SB % 4 == 0 && KS % PFB == 0 && NW >= 4, "pipeline shape");
  __shared__ __attribute__((aligned(1024))) bf16 As[NBUF][SB * BLK];
  static_assert(32 * PB * TN * 4 <= (int)sizeof(As), "an epilogue pass must fit the stage buffers");

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n_blocks = (a.N + 31) >> 5, n_nt = (n_blocks + NW * CB - 1) / (NW * CB);
  const int m_blocks = (a.M + 31) >> 5, n_mt = (m_blocks + FM - 1) / FM;
  const int S = a.splits;
  const int t = xcd_remap(blockIdx.x, n_mt * n_nt * S);
  const int mt = t % n_mt, rest = t / n_mt;
  const int sp = rest % S, nt = rest / S;
  const int ks16 = a.Kp >> 4;
  const int units = ks16 / (KS * NBUF), per = (units + S - 1) / S;
  const int kb = min(units, sp * per) * (KS * NBUF), ke = min(units, sp * per + per) * (KS * NBUF);
  const int n_st = (ke - kb) / KS;  // a multiple of NBUF
  // this wave's weight blocks (past N: a valid block whose columns are never stored)
  const bf16* bp[CB];
  static_for<0, CB>([&](auto c) {
    bp[c] = (const bf16*)a.B + (size_t)min((nt * NW + wave) * CB + (int)decltype(c)::value, n_blocks - 1) * a.bstride +
            lane * 8;
  });
  const bf16* __restrict__ Ab = (const bf16*)a.A;
  float* T_ = (float*)&As[0][0];
  const int m0 = mt * FM * 32, n0 = nt * TN;

  auto body = [&](auto d_c) {
    constexpr int D = decltype(d_c)::value;  // DMAs per stage issued by this wave
    auto dma = [&](auto buf, int st) {
      static_for<0, D>([&](auto d) {
        const int q = wave + 4 * decltype(d)::value, mb = q / KS, j = q % KS;
        const int k = min(kb + st * KS + j, ks16 - 1);
        const int blk = min(mt * FM + mb, m_blocks - 1);  // rows past M: a valid block, never stored
        const bf16* src = Ab + (size_t)blk * a.astride + (size_t)k * BLK + lane * 8;
        __builtin_amdgcn_global_load_lds((const void*)src,
                                         (__attribute__((address_space(3))) void*)&As[buf][q * BLK], 16, 0, 0);
      });
    };
    bf16x8 rb[PFB][CB];
    auto load_b = [&](auto slot, int st, int j) {
      const int k = min(kb + st * KS + j, ks16 - 1);
      static_for<0, CB>([&](auto c) {
        const bf16* src = bp[c] + (size_t)k * BLK;
        bf16x8 v;
        asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(v) : "v"(src) : "memory");
        rb[slot][c] = v;
      });
    };
    f32x16 acc[FM][CB];
    static_for<0, FM>([&](auto i) { static_for<0, CB>([&](auto c) { acc[i][c] = f32x16{}; }); });
    static_for<0, NBUF - 1>([&](auto b) {
      dma(b, b);
      __builtin_amdgcn_sched_barrier(0);
    });
    static_for<0, PFB>([&](auto j) { load_b(std::integral_constant<int, decltype(j)::value>{}, 0, j); });
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the loop's waits count from a full ring
    __builtin_amdgcn_sched_barrier(0);
    for (int st0 = 0; st0 < n_st; st0 += NBUF) {
      static_for<0, NBUF>([&](auto u) {
        constexpr int U = decltype(u)::value;
        const int st = st0 + U;
        // Loads complete in order.  Stage st's activations come from the DMA at the top of stage
        // st - NBUF + 1, after which NBUF - 1 stages of weight loads (CB KS each) and NBUF - 2
        // DMAs were issued.  k step j's weights were loaded PFB steps earlier; after them came
        // the CB (PFB - 1) weight loads of the steps between and, when a stage top lies between,
        // its DMAs.
        constexpr int WAIT_A = CB * KS * (NBUF - 1) + D * (NBUF - 2);
        static_assert(WAIT_A <= 63, "vmcnt range");
        asm volatile("s_waitcnt vmcnt(%0) lgkmcnt(0)\n\ts_barrier" ::"n"(WAIT_A) : "memory");
        dma(std::integral_constant<int, (U + NBUF - 1) % NBUF>{}, st + NBUF - 1);
        __builtin_amdgcn_sched_barrier(0);
        bf16x8 af[AFB][FM];
        if constexpr (AFB == 2) {
          static_for<0, FM>([&](auto i) {
            af[0][i] = *(const bf16x8*)(&As[U][((int)decltype(i)::value * KS) * BLK + lane * 8]);
          });
        }
        static_for<0, KS>([&](auto j) {
          constexpr int J = decltype(j)::value;
          constexpr int slot = (U * KS + J) % PFB;
          constexpr int CUR = AFB == 2 ? (J & 1) : 0;
          if constexpr (AFB == 2) {  // the next k step's fragments, read while these MFMAs run
            if constexpr (J + 1 < KS) {
              static_for<0, FM>([&](auto i) {
                af[(J + 1) & 1][i] = *(const bf16x8*)(&As[U][((int)decltype(i)::value * KS + J + 1) * BLK + lane * 8]);
              });
            }
          } else {
            static_for<0, FM>([&](auto i) {
              af[0][i] = *(const bf16x8*)(&As[U][((int)decltype(i)::value * KS + J) * BLK + lane * 8]);
            });
          }
          constexpr int WAIT_B = CB * (PFB - 1) + (J < PFB ? D : 0);
          asm volatile("s_waitcnt vmcnt(%0)" ::"n"(WAIT_B) : "memory");
          __builtin_amdgcn_sched_barrier(0);
          static_for<0, FM>([&](auto i) {
            static_for<0, CB>([&](auto c) {
              acc[i][c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[CUR][i], rb[slot][c], acc[i][c], 0, 0, 0);
            });
          });
          load_b(std::integral_constant<int, slot>{}, st + (J + PFB) / KS, (J + PFB) % KS);
          __builtin_amdgcn_sched_barrier(0);
        });
      });
    }
    // the ring's last (unused) loads land before any of its registers can be reused
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
    for (int p = 0; p < PFB; ++p)
#pragma unroll
      for (int c = 0; c < CB; ++c) asm volatile("" : "+v"(rb[p][c]));

    // ---- epilogue, PB row blocks per pass through the stage buffers
    constexpr bool paired = EPI == EPI_SWIGLU || EPI == EPI_QKV;
    constexpr int W = paired ? 16 : 8;
    static_for<0, NPASS>([&](auto p_c) {
      constexpr int PS = decltype(p_c)::value;
      constexpr int NB = PS * PB + PB <= FM ? PB : FM - PS * PB;  // row blocks in this pass
      __syncthreads();  // every wave's DMAs have landed and the buffers' last readers are done
      static_for<0, NB>([&](auto i) {
        static_for<0, CB>([&](auto c) {
          static_for<0, 16>([&](auto r) {
            constexpr int R = decltype(r)::value;
            const int row = (int)decltype(i)::value * 32 + 8 * (R / 4) + 4 * (lane >> 5) + (R % 4);
            T_[row * TN + (wave * CB + (int)decltype(c)::value) * 32 + (lane & 31)] =
                acc[PS * PB + decltype(i)::value][decltype(c)::value][R];
          });
        });
      });
      __syncthreads();
      constexpr int ITEMS = 32 * NB * (TN / W);
      for (int it = tid; it < ITEMS; it += 64 * NW) {
        const int row = it / (TN / W), col = (it % (TN / W)) * W;
        const int m = m0 + PS * PB * 32 + row, nc = n0 + col;
        if (m >= a.M || nc >= a.N) continue;  // N % 16 == 0: a group is wholly inside or outside
        float v[W];
#pragma unroll
        for (int e = 0; e < W; e += 4) *(f32x4*)&v[e] = *(const f32x4*)&T_[row * TN + col + e];
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
    });
  };
  if (wave < 4)
    body(std::integral_constant<int, DW>{});
  else
    body(std::integral_constant<int, 0>{});
}

// NW-wave variant for 161..384 rows: the tile is 32 FM rows (FM = 5 or 6) x 32 NW columns, each
// wave owning one 32-column weight block over all FM row blocks, so no weight fragment is loaded
// twice and two row tiles fill the GPU where 288 x 128 tiles leave part of it idle.  Activations go
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

// The 160-row tiles (192-row tiles from 321 to 384 rows, so that two row tiles still hold every
// row) are taken in two cases:
//  * six waves (192 columns), unsplit or split two ways over K, when that fills 3/4 of the GPU
//    or more in one pass (a 7B-shape step's gate/up projection: 2 x 115 = 230 workgroups; QKV:
//    2 x 64 x 2 = 256);
//  * four waves (128 columns) for narrow projections (N <= 4096) split four ways over K (the
//    output and down projections: 2 x 32 x 4 = 256 workgroups), which write half the fp32
//    partial sums of the 8-way split the 288 x 128 tile needs to fill the GPU.
constexpr int C6_NW = 6;
// 32-row blocks per row tile: 5 for 6..10 blocks, 6 for 11..12, else none.
static int c6_fm(int M) {
  const int mb = (M + 31) / 32;
  return mb > 5 && mb <= 10 ? 5 : mb > 10 && mb <= 12 ? 6 : 0;
}
static int c6_narrow(int M, int N, int Kp) {
  const int fm = c6_fm(M), nb = (N + 31) / 32, units = Kp / 256;
  if (!fm || nb > 128 || units < 4) return 0;
  const int S = 4, per = (units + S - 1) / S;
  return (units + per - 1) / per;
}
// Split-K factor of the six-wave plan: 1 or 2, whichever puts 192..256 workgroups in one pass
// (0: the plan does not fit).
static int c6_wide_splits(int M, int N, int Kp) {
  const int fm = c6_fm(M);
  if (!fm) return 0;
  const int mb = (M + 31) / 32, nb = (N + 31) / 32;
  const int tiles = ((mb + fm - 1) / fm) * ((nb + C6_NW - 1) / C6_NW);
  if (tiles >= 192 && tiles <= 256) return 1;
  if (2 * tiles >= 192 && 2 * tiles <= 256 && Kp / 256 >= 2) return 2;
  return 0;
}
static bool use_c6(int epi, const GemmArgs& a) {
  const int fm = c6_fm(a.M);
  if (!fm || (fm == 6 && epi == EPI_STORE_F32 && a.splits == 1)) return false;
  if (a.splits > 1 && a.splits == c6_narrow(a.M, a.N, a.Kp)) return true;
  return a.splits == c6_wide_splits(a.M, a.N, a.Kp);
}

template <int FM>
static hipError_t gemm32c_launch_fm(int epi, const GemmArgs& a, hipStream_t s) {
  const int mb = (a.M + 31) / 32, nb = (a.N + 31) / 32;
  if (a.splits > 1 && a.splits == c6_narrow(a.M, a.N, a.Kp)) {  // narrow: four-wave FM x 4 block tile
    const dim3 grid(((mb + FM - 1) / FM) * ((nb + 3) / 4) * a.splits);
    hipLaunchKernelGGL((gemm32c_kernel<FM, 4, EPI_STORE>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
  }
  const dim3 grid(((mb + FM - 1) / FM) * ((nb + C6_NW - 1) / C6_NW) * a.splits), block(64 * C6_NW);
  if (a.splits > 1) {  // partial sums only: one instance serves every epilogue
    hipLaunchKernelGGL((gemm32c_kernel<FM, C6_NW, EPI_STORE>), grid, block, 0, s, a);
    return hipGetLastError();
  }
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL((gemm32c_kernel<FM, C6_NW, EPI_STORE>), grid, block, 0, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL((gemm32c_kernel<FM, C6_NW, EPI_RESID>), grid, block, 0, s, a); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm32c_kernel<FM, C6_NW, EPI_SWIGLU>), grid, block, 0, s, a); break;
    case EPI_QKV: hipLaunchKernelGGL((gemm32c_kernel<FM, C6_NW, EPI_QKV>), grid, block, 0, s, a); break;
    case EPI_STORE_F32:
      if constexpr (FM == 5) {
        hipLaunchKernelGGL((gemm32c_kernel<FM, C6_NW, EPI_STORE_F32>), grid, block, 0, s, a);
        break;
      }
      return hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

static hipError_t gemm32c_launch(int epi, const GemmArgs& a, hipStream_t s) {
  return c6_fm(a.M) == 6 ? gemm32c_launch_fm<6>(epi, a, s) : gemm32c_launch_fm<5>(epi, a, s);
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

// The wide 288 x 256 tile where it takes less time than the 288 x 128 one, whole passes of 256
// workgroups compared with a wide tile measured at 1.8 times a narrow one (about 132 against
// 76 us at K = 4096): at 2264 rows gate/up takes 3 wide passes instead of 6 narrow ones, and
// at 518 one instead of 2.  Where one pass of wide tiles over the first columns and narrow
// tiles for the rest cost less than either alone (QKV at 2264 rows: 1 wide pass over 8192
// columns and 1 narrow pass over 4096, against 3 narrow or 2 wide passes), the launch is split
// there.  The output and down projections at 2264 rows stay narrow.  Unsplit only.
// Returns 0 (narrow), 1 (wide) or the first narrow column of a split launch.
static int wide_plan(int epi, const GemmArgs& a) {
  if (a.splits != 1 || a.col0 != 0 || epi == EPI_STORE_F32 || fm_for(a.M) != 9 || a.M <= 32 * 12) return 0;
  const int mb = (a.M + 31) / 32, nb = (a.N + 31) / 32, n_mt = (mb + 8) / 9;
  auto passes = [](long t) { return (t + 255) / 256; };
  const long cost_n = passes((long)n_mt * ((nb + 3) / 4)) * 10;
  const long cost_w = passes((long)n_mt * ((nb + 7) / 8)) * 18;
  const int wblocks = (256 / n_mt) * 8;  // column blocks of one pass of wide tiles
  const long cost_h = wblocks > 0 && wblocks < nb ? 18 + passes((long)n_mt * ((nb - wblocks + 3) / 4)) * 10 : cost_w + 1;
  if (cost_h < cost_w && cost_h < cost_n) return wblocks * 32;
  return cost_w < cost_n ? 1 : 0;
}

static hipError_t gemm32w_launch(int epi, const GemmArgs& a, hipStream_t s) {
  const int mb = (a.M + 31) / 32, nb = (a.N + 31) / 32;
  constexpr int FM = 9, NW = 8, CB = 1;
  const dim3 grid(((mb + FM - 1) / FM) * ((nb + NW * CB - 1) / (NW * CB)) * a.splits), block(64 * NW);
  switch (epi) {
    case EPI_STORE: hipLaunchKernelGGL((gemm32w_kernel<FM, NW, CB, EPI_STORE>), grid, block, 0, s, a); break;
    case EPI_RESID: hipLaunchKernelGGL((gemm32w_kernel<FM, NW, CB, EPI_RESID>), grid, block, 0, s, a); break;
    case EPI_SWIGLU: hipLaunchKernelGGL((gemm32w_kernel<FM, NW, CB, EPI_SWIGLU>), grid, block, 0, s, a); break;
    case EPI_QKV: hipLaunchKernelGGL((gemm32w_kernel<FM, NW, CB, EPI_QKV>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

static hipError_t gemm_dispatch_bf16(int epi, const GemmArgs& a, hipStream_t s) {
  if (a.astride <= 0 || a.Kp % 256 != 0 || a.astride < (long)a.Kp * 32 || a.bstride < (long)a.Kp * 32)
    return hipErrorInvalidValue;
  hipError_t e;
  if (use_c6(epi, a)) {
    e = gemm32c_launch(epi, a, s);
    if (e != hipSuccess || a.splits <= 1 || a.partials_only) return e;
    return reduce_launch<bf16>(epi, a, s);
  }
  if (const int plan = wide_plan(epi, a)) {
    if (plan == 1) return gemm32w_launch(epi, a, s);
    // columns [0, plan) on wide tiles, the rest on 288 x 128 tiles
    GemmArgs aw = a, an = a;
    aw.N = plan;
    an.N = a.N - plan;
    an.col0 = plan;
    an.B = (const bf16*)a.B + (size_t)(plan / 32) * a.bstride;
    e = gemm32w_launch(epi, aw, s);
    if (e != hipSuccess) return e;
    return gemm32_launch<9, true>(epi, an, s);
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
    if (const int S = c6_wide_splits(M, N, Kp)) return S;
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

}  // namespace af
