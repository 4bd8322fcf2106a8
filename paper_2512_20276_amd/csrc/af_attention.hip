// gfx950 kernels of the segment-aware attention (Alg. 2 VarlenAttention): every packed row
// attends only to its own request's region of the ring, causally inside a prefill segment and
// over the full history for a decode row.
#include "af_device.h"

namespace af {

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

// ROWS (1 or 2) single-row segments per workgroup of NWG waves: tiles first .. first + ROWS - 1
// (those that exist), each on NWG / ROWS waves.  Two per workgroup halve the workgroups a packed
// step's decode rows take next to its query tiles.  Either way a row is computed as ATTN_WAVES
// virtual waves (virtual wave v takes chunks v, v + ATTN_WAVES, ..; a wave of a row on four
// waves runs two of them one after the other) merged in virtual-wave order, so the result does
// not depend on how many rows share the workgroup or how many waves it has.
template <typename T, int HD, int ROWS, int NWG = ATTN_WAVES>
__device__ __forceinline__ void attention_decode_rows(const AttnArgs& a, int first, int h) {
  constexpr int VEC = Chunk<T>::N;  // elements per 16 bytes
  constexpr int DG = HD / VEC;      // 16-byte chunks per key row
  constexpr int KH2 = DG / 2;       // chunks per half row (two lanes per key for the scores)
  constexpr int KG = 64 / DG;       // value key groups (lane / DG)
  constexpr int KPL = 32 / KG;      // values: keys per lane per 32-key chunk
  static_assert(DG % 2 == 0 && DG <= 64 && 64 % DG == 0 && 32 % KG == 0, "head_dim");
  static_assert(ROWS == 1 || ROWS == 2, "rows per workgroup");
  constexpr int VW = ATTN_WAVES;  // virtual waves per row
  constexpr int NW = NWG / ROWS;  // waves per row
  static_assert(VW % NW == 0, "virtual waves per wave");
  __shared__ float wm[ROWS][VW], wl[ROWS][VW];
  __shared__ __attribute__((aligned(16))) float wo[ROWS][VW][HD];
  __shared__ __attribute__((aligned(16))) uint4 qs[ROWS][DG];
  const int tid = threadIdx.x, lane = tid & 63, wave0 = tid >> 6;
  const int sub = ROWS == 1 ? 0 : wave0 / NW, wave = ROWS == 1 ? wave0 : wave0 % NW;  // row, wave within it
  const bool live = ROWS == 1 || first + sub < a.n_tiles;  // an odd count leaves the last half idle
  const int seg_i = a.tiles[2 * (live ? first + sub : first)];
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
// the current one is processed from LDS (its load overlaps the current tile's arithmetic).
// The segment's key tiles are split between two key groups (group g takes tiles g, g + 2,
// g + 4, ..), each with a softmax state of its own, and group 1's state is merged into group
// 0's at the end.  With NWG = 8 waves the two groups run at once, four waves each, with LDS
// buffers of their own; with NWG = 4 one set of waves runs group 0 and then group 1, parking
// group 0's state in LDS.  Both do the same arithmetic in the same order, so a row's result
// does not depend on which of the two ran it.
template <typename T, int HD>
struct AttnLds {
  static constexpr int VEC = Chunk<T>::N;
  static constexpr int KROW = HD + VEC;        // padded key row (elements)
  static constexpr int VROW = ATTN_BKV + VEC;  // padded transposed-value row
  static constexpr int K_ELEMS = ATTN_BKV * KROW, V_ELEMS = HD * VROW;
  static constexpr int GROUP_BYTES = (K_ELEMS + V_ELEMS) * (int)sizeof(T);
  static constexpr int MERGE_BYTES = 4 * 64 * (2 + 4 * (HD / 16)) * (int)sizeof(float);  // 4 waves' states
  // LDS of a query-tile workgroup: two groups' buffers (8 waves; the merge reuses them), or one
  // group's buffers and the parked state (4 waves)
  static constexpr int bytes(int nwg) { return nwg == 8 ? 2 * GROUP_BYTES : GROUP_BYTES + MERGE_BYTES; }
};

// The merge of key group 1's state (m1, l1, o1) into group 0's (m0, l0, o0).
__device__ __forceinline__ void merge_state(float& m0, float& l0, float m1, float l1, float& f0, float& f1) {
  const float M = fmaxf(m0, m1);
  f0 = m0 == -INFINITY ? 0.f : exp2f(m0 - M);
  f1 = m1 == -INFINITY ? 0.f : exp2f(m1 - M);
  l0 = __builtin_fmaf(l0, f0, l1 * f1);
  m0 = M;
}

template <typename T, int HD, int NWG>
__device__ __forceinline__ void attention_prefill_tile(const AttnArgs& a, int tile, int h, char* smem) {
  typedef AttnLds<T, HD> L;
  constexpr int VEC = L::VEC, KROW = L::KROW, VROW = L::VROW;
  constexpr int KST = HD / 32;              // MFMA k steps over the head dimension
  constexpr int DB = HD / 16;               // 16-dim output blocks
  constexpr int CPR = HD / VEC;             // 16-byte chunks per key row
  constexpr int NCH = ATTN_BKV * CPR / 256; // chunks of K (and of V) per thread per tile
  constexpr int NPG = NWG / 4;              // key groups running at once
  static_assert((ATTN_BKV * CPR) % 256 == 0 && (NWG == 4 || NWG == 8), "tile shape");
  typedef typename Mma<T>::frag frag;

  const int lane = threadIdx.x & 63, pgrp = threadIdx.x >> 8, wave = (threadIdx.x >> 6) & 3;
  const int tid = threadIdx.x & 255;  // position within the key group
  T* const Ks = (T*)smem + (size_t)pgrp * (L::K_ELEMS + L::V_ELEMS);
  T* const Vt = Ks + L::K_ELEMS;
  const int lr = lane & 15, lg = lane >> 4;
  const int seg_i = a.tiles[2 * tile], i0 = a.tiles[2 * tile + 1];
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


  // One tile's keys and values in registers.  Keys: thread t holds 16-byte chunk t % CPR of
  // keys t / CPR + KR j (row-major LDS writes, one key row per CPR lanes).  Values: thread t
  // holds KPT consecutive keys (t % KGV) * KPT .. of dim chunk t / KGV, so that after a
  // transpose in registers each dim's KPT keys go to LDS as one contiguous write.
  constexpr int KR = 256 / CPR;          // key rows per pass
  constexpr int KPT = NCH;               // values: keys per thread
  constexpr int KGV = ATTN_BKV / KPT;    // values: key groups
  static_assert(KGV * CPR == 256, "value mapping");
  // Keys past kv_end are loaded from the last visible key (unconditional loads, so nothing waits
  // for them until the tile is parked) and replaced by zeros when the tile is parked.
  uint4 kreg[NCH], vreg[NCH];
  const int kc = tid % CPR, kr = tid / CPR;
  const int vg = tid % KGV, vc = tid / KGV;
  auto load_tile = [&](int kb0) {
#pragma unroll
    for (int j = 0; j < NCH; ++j) {
      const int key = min(kb0 + kr + KR * j, kv_end - 1);
      kreg[j] = *(const uint4*)(Kg + (size_t)key * HD + kc * VEC);
      const int vkey = min(kb0 + vg * KPT + j, kv_end - 1);
      vreg[j] = *(const uint4*)(Vg + (size_t)vkey * HD + vc * VEC);
    }
  };
  const int n_kt = (kv_end + ATTN_BKV - 1) / ATTN_BKV;
  const int n_it = (n_kt + 1) / 2;  // both groups run the same iterations (and barriers)
  f32x4 oacc[DB];
  float m_run = -INFINITY, l_run = 0.f;
  float* const park = (float*)(smem + L::GROUP_BYTES) + (size_t)wave * (2 + 4 * DB) * 64 + lane;
  for (int grp = pgrp; grp < 2; grp += NPG) {
#pragma unroll
    for (int d = 0; d < DB; ++d) oacc[d] = f32x4{0.f, 0.f, 0.f, 0.f};
    m_run = -INFINITY;
    l_run = 0.f;
    load_tile(grp * ATTN_BKV);
    for (int it = 0; it < n_it; ++it) {
      const int kt = 2 * it + grp;
      const int kb0 = kt * ATTN_BKV;
      // ---- park the tile in LDS: keys row-major, values transposed
      __syncthreads();  // the previous tile's LDS reads are done
#pragma unroll
      for (int j = 0; j < NCH; ++j)
        *(uint4*)(&Ks[(kr + KR * j) * KROW + kc * VEC]) = kb0 + kr + KR * j < kv_end ? kreg[j] : zero4();
      {
        T vt[NCH][VEC];
#pragma unroll
        for (int j = 0; j < NCH; ++j) {
          const uint4 v = kb0 + vg * KPT + j < kv_end ? vreg[j] : zero4();
          __builtin_memcpy(vt[j], &v, 16);
        }
#pragma unroll
        for (int e = 0; e < VEC; ++e) {
          T col[KPT];
#pragma unroll
          for (int j = 0; j < KPT; ++j) col[j] = vt[j][e];
          T* dst = &Vt[(vc * VEC + e) * VROW + vg * KPT];
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
            const T* vrow = &Vt[(d * 16 + lr) * VROW + c * 32 + lg * 4];
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
    if (NWG == 4 && grp == 0) {  // park group 0's state for the merge
      park[0] = m_run;
      park[64] = l_run;
#pragma unroll
      for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int e = 0; e < 4; ++e) park[(2 + 4 * d + e) * 64] = oacc[d][e];
    }
  }

  // ---- merge key group 1 into group 0 (per lane: the same query and output dims in both)
  constexpr int NF = 2 + 4 * DB;  // m, l, the output accumulators
  static_assert(4 * 64 * NF * sizeof(float) <= (size_t)L::GROUP_BYTES && 4 * 64 * NF * sizeof(float) <= (size_t)L::MERGE_BYTES,
                "merge buffer");
  if constexpr (NWG == 8) {
    float* mb = (float*)smem + (size_t)wave * NF * 64 + lane;
    __syncthreads();  // every wave is done with the key/value buffers
    if (pgrp == 1) {
      mb[0] = m_run;
      mb[64] = l_run;
#pragma unroll
      for (int d = 0; d < DB; ++d)
#pragma unroll
        for (int e = 0; e < 4; ++e) mb[(2 + 4 * d + e) * 64] = oacc[d][e];
    }
    __syncthreads();
    if (pgrp == 1) return;
    float f0, f1;
    merge_state(m_run, l_run, mb[0], mb[64], f0, f1);
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int e = 0; e < 4; ++e) oacc[d][e] = __builtin_fmaf(oacc[d][e], f0, mb[(2 + 4 * d + e) * 64] * f1);
  } else {  // this lane's state is group 1's; group 0's is parked
    float m0 = park[0], l0 = park[64], f0, f1;
    merge_state(m0, l0, m_run, l_run, f0, f1);
    l_run = l0;
#pragma unroll
    for (int d = 0; d < DB; ++d)
#pragma unroll
      for (int e = 0; e < 4; ++e) oacc[d][e] = __builtin_fmaf(park[(2 + 4 * d + e) * 64], f0, oacc[d][e] * f1);
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
// (ordered longest first), the rest single-row segments.  The grid is one-dimensional with the
// head varying fastest, block = item * n_heads + head: every head of the longest query tile is
// dispatched first and the short items last, and the query tiles of one head (32 blocks apart
// at 32 heads) land on the same XCD, whose L2 then serves the segment's keys to all of them.
// Items [0, n_multi) of the query-tile instance are the query tiles, its other items pairs of
// single-row tiles (n_multi + 2 (item - n_multi) and the next); the decode-only instance takes
// one single-row tile per item (n_multi + item), on all of its waves.
template <typename T, int HD, bool PREFILL>
__global__ __launch_bounds__(64 * ATTN_WAVES, !PREFILL ? 4 : 2) void attention_kernel(AttnArgs a) {
  const int b = blockIdx.x / a.n_heads, h = blockIdx.x % a.n_heads;
  if constexpr (PREFILL) {
    __shared__ __attribute__((aligned(16))) char smem[AttnLds<T, HD>::bytes(8)];
    if (b < a.n_multi)
      attention_prefill_tile<T, HD, 8>(a, b, h, smem);
    else
      attention_decode_rows<T, HD, 2>(a, a.n_multi + 2 * (b - a.n_multi), h);
  } else {
    attention_decode_rows<T, HD, 1>(a, a.n_multi + b, h);
  }
}

// Four-wave workgroups for steps whose decode rows would more than fill the GPU beside the query
// tiles (many pipelines, long action chunks): work item b < n_multi is query tile b (its key
// groups one after the other), any other the single-row tile b.  Several such workgroups share
// a CU, and the blocks alternate between the two kinds in groups of eight (one block per XCD
// each), so the decode rows' key and value streams run beside the latency-bound query tiles from
// the start instead of after them.  Within each kind the order is (work item, head) with the
// head fastest, so a query tile's XCD is still set by its head.  The results are those of the
// eight-wave instances bit for bit.
template <typename T, int HD>
__global__ __launch_bounds__(256, 3) void attention_kernel4(AttnArgs a) {
  const int nb_t = a.n_multi * a.n_heads, nb_d = (a.n_tiles - a.n_multi) * a.n_heads;
  const int inter = min(nb_t, nb_d) / 8 * 8;  // blocks of each kind that alternate
  const int x = blockIdx.x;
  int item;  // (work item) * n_heads + head
  if (x < 2 * inter) {
    const int g = x >> 4, r = x & 15;
    item = r < 8 ? g * 8 + r : nb_t + g * 8 + (r - 8);
  } else {  // the rest: query tiles left over, then decode rows
    const int rest = x - 2 * inter, t_left = nb_t - inter;
    item = rest < t_left ? inter + rest : nb_t + inter + (rest - t_left);
  }
  const int b = item / a.n_heads, h = item % a.n_heads;
  __shared__ __attribute__((aligned(16))) char smem[AttnLds<T, HD>::bytes(4)];
  if (b < a.n_multi)
    attention_prefill_tile<T, HD, 4>(a, b, h, smem);
  else
    attention_decode_rows<T, HD, 1, 4>(a, b, h);
}

// Query tiles and decode rows share one launch: eight-wave workgroups (two decode rows each,
// after the query tiles) while the decode rows fit one pass over the CUs and the whole launch
// fits 1.4 passes, else four-wave workgroups (one decode row each, alternating with the query
// tiles), two of which share a CU; a step without query tiles takes the decode-only instance.
// Where the decode rows are many, overlapping their key and value streams with the query tiles
// pays more than the query tiles' own two concurrent key groups (measured on the 8-pipeline
// step, and on a 276- or 512-row prefill beside 7 to 15 decode rows); just past one pass the
// eight-wave launch's second pass is short and the query tiles' latency decides.
template <typename T, int HD>
static void attention_launch(const AttnArgs& a0, int n_tiles, hipStream_t s) {
  AttnArgs a = a0;
  a.n_tiles = n_tiles;
  const dim3 block(64 * ATTN_WAVES);
  const int n_single = n_tiles - a.n_multi, n_pairs = (n_single + 1) / 2;
  if (a.n_multi == 0) {
    hipLaunchKernelGGL((attention_kernel<T, HD, false>), dim3(n_tiles * a.n_heads), block, 0, s, a);
  } else if ((long)n_pairs * a.n_heads <= 256 && (long)(a.n_multi + n_pairs) * a.n_heads * 5 <= 256 * 7) {
    hipLaunchKernelGGL((attention_kernel<T, HD, true>), dim3((a.n_multi + n_pairs) * a.n_heads), block, 0, s, a);
  } else {
    hipLaunchKernelGGL((attention_kernel4<T, HD>), dim3(n_tiles * a.n_heads), dim3(256), 0, s, a);
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

}  // namespace af
