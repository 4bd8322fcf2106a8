// Weights, scratch activations and the orchestration of the packed forward (Alg. 1 head,
// Alg. 2 per layer).  Host code only: argument checking, the per-call step descriptor
// (segment table, per-row slot/position, attention work tiles, emitting rows) and the
// kernel sequence.  Every step of the path runs in the kernels of af_gemm.hip, af_attention.hip
// and af_kernels.hip.
#include <algorithm>
#include <cmath>
#include <cstring>
#include <new>
#include <numeric>
#include <vector>

#include "af_internal.h"

using namespace af;

namespace {

// Projection weights are stored fragment-tiled for the GEMM (K padded to a multiple of 32).
struct Layer {
  void* attn_norm = nullptr;
  void* wqkv = nullptr;  // [3d, d]: q, k, v rows, each head in rotary-pair 16-row block order
  void* wo = nullptr;    // [d, d]
  void* mlp_norm = nullptr;
  void* wgu = nullptr;   // [2 d_ff, d]: gate/up rows in alternating 16-row blocks
  void* wdown = nullptr; // [d, d_ff]
};

// K of the fragment-tiled weights: padded so the GEMM's k loop has no partial unrolled block.
inline int padk(int k) { return (k + gemm_k_align() - 1) / gemm_k_align() * gemm_k_align(); }

struct StageBuf {  // pinned staging for one descriptor upload
  int32_t* host = nullptr;
  size_t cap = 0;  // int32 elements
  hipEvent_t done = nullptr;
  bool pending = false;
};

struct TimedLaunch {
  int cls;
  hipEvent_t start, stop;
};

}  // namespace

struct af_weights {
  af_model_desc d{};
  size_t es = 2;
  std::vector<void*> allocs;
  void* embed = nullptr;
  void* final_norm = nullptr;
  void* lm_head = nullptr;
  std::vector<Layer> layers;

  float* rope_cs = nullptr;  // [rope_cap][hd/2][2]
  int rope_cap = 0;

  // scratch activations, grown on demand.  bf16: the GEMM inputs xn, attn, act and emit_norm are
  // fragment-tiled (32-row blocks xs_D / xs_F elements apart, zero-filled once so the K padding
  // stays zero); fp32: row-major with the padded strides ldD / ldF.  q is row-major in both.
  int ws_M = 0, ws_emit = 0;
  int ldD = 0, ldF = 0;
  long xs_D = 0, xs_F = 0;
  void *xn = nullptr, *q = nullptr, *attn = nullptr, *act = nullptr, *emit_norm = nullptr;
  float* logits_ws = nullptr;
  int32_t* tokens_ws = nullptr;
  int32_t* dev_err = nullptr;

  float* partial = nullptr;  // split-K partial sums
  size_t partial_cap = 0;    // floats

  int32_t* desc_dev = nullptr;
  size_t desc_cap = 0;
  StageBuf stage[4];
  int stage_next = 0;

  uint32_t options = 0;
  uint32_t timing_mask = 0;
  std::vector<TimedLaunch> timed;
  std::vector<hipEvent_t> event_pool;
};

namespace {

// Device workspace of one forward call.  The allocating entry points take it from the weights
// object (grown on demand, `grow` set); the no-allocation entry point carves it from a fixed
// buffer (`grow` null: a split-K partial buffer that is too small is an error, not a resize).
// `timing` is the weights object whose timing mask applies, or null for no timing.
struct Ws {
  af_weights* grow = nullptr;
  af_weights* timing = nullptr;
  void *xn = nullptr, *q = nullptr, *attn = nullptr, *act = nullptr, *emit_norm = nullptr;
  float* logits = nullptr;  // fp32 logits of the emitting rows when the caller passes none
  int32_t* desc = nullptr;  // the uploaded step tables
  const float* rope = nullptr;
  float* partial = nullptr;
  size_t partial_cap = 0;   // floats
};

af_status dev_alloc(af_weights* w, void** p, size_t bytes) {
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    set_error("hipMalloc(%zu) failed: %s", bytes, hipGetErrorString(e));
    *p = nullptr;
    return AF_ERR_OOM;
  }
  w->allocs.push_back(*p);
  return AF_OK;
}

void dev_free(af_weights* w, void* p) {
  if (!p) return;
  auto it = std::find(w->allocs.begin(), w->allocs.end(), p);
  if (it != w->allocs.end()) w->allocs.erase(it);
  (void)hipFree(p);
}

af_status check_model_desc(const af_model_desc& d) {
  if (d.dtype != AF_BF16 && d.dtype != AF_F32) {
    set_error("model dtype must be AF_BF16 or AF_F32");
    return AF_ERR_INVALID_ARG;
  }
  if (d.n_layers < 0 || d.d_model <= 0 || d.n_heads <= 0 || d.vocab <= 0 || d.d_ff <= 0) {
    set_error("model dimensions must be positive");
    return AF_ERR_INVALID_ARG;
  }
  if (d.n_kv_heads != d.n_heads || (d.head_dim != 64 && d.head_dim != 128) || d.d_model != d.n_heads * d.head_dim ||
      d.d_model % 32 != 0 || d.d_ff % 16 != 0) {
    set_error("unsupported model shape: need n_kv_heads == n_heads, head_dim in {64,128}, d_model == heads*head_dim, "
              "d_model %% 32 == 0, d_ff %% 16 == 0");
    return AF_ERR_UNSUPPORTED;
  }
  if (!(d.rms_eps >= 0.f) || !(d.rope_theta > 0.f)) {
    set_error("rms_eps must be >= 0 and rope_theta > 0");
    return AF_ERR_INVALID_ARG;
  }
  return AF_OK;
}

af_status check_ring_matches(const af_weights* w, const af_ring* r, int min_layers) {
  if (!r) {
    set_error("NULL ring");
    return AF_ERR_INVALID_ARG;
  }
  if (!r->kv) {
    set_error("bookkeeping-only ring (n_layers == 0) cannot run the forward");
    return AF_ERR_INVALID_ARG;
  }
  if (r->d.n_layers < min_layers || r->d.n_kv_heads != w->d.n_kv_heads || r->d.head_dim != w->d.head_dim ||
      r->d.dtype != w->d.dtype) {
    set_error("ring (layers %d, heads %d, head_dim %d, dtype %d) does not match the model (layers %d, heads %d, "
              "head_dim %d, dtype %d)",
              r->d.n_layers, r->d.n_kv_heads, r->d.head_dim, r->d.dtype, min_layers, w->d.n_kv_heads, w->d.head_dim,
              w->d.dtype);
    return AF_ERR_INVALID_ARG;
  }
  return AF_OK;
}

// Segment rules shared by every entry point that takes a segment table.
af_status check_segments(const af_ring* ring, const af_segment* segs, int n_seg, int M) {
  if (!segs || n_seg <= 0 || n_seg > MAX_SEGMENTS) {
    set_error("segment table: need 1..%d segments (got %d)", MAX_SEGMENTS, n_seg);
    return AF_ERR_INVALID_ARG;
  }
  if (M <= 0) {
    set_error("M must be positive (got %d)", M);
    return AF_ERR_INVALID_ARG;
  }
  std::vector<int> order(n_seg);
  std::vector<char> slot_used(ring->d.n_slots, 0);
  for (int i = 0; i < n_seg; ++i) {
    const af_segment& s = segs[i];
    order[i] = i;
    if (s.q_len <= 0 || s.q_start < 0 || (int64_t)s.q_start + s.q_len > M || s.reserved != 0 ||
        (s.flags & ~AF_SEG_EMIT) != 0) {
      set_error("segment %d: rows [%d, %d) outside [0, %d) or bad flags/reserved", i, s.q_start, s.q_start + s.q_len, M);
      return AF_ERR_INVALID_ARG;
    }
    if (s.slot < 0 || s.slot >= ring->d.n_slots || s.pos0 < 0 || (int64_t)s.pos0 + s.q_len > ring->d.max_pos) {
      set_error("segment %d: slot %d / positions [%d, %d) outside the ring (%d slots x %d)", i, s.slot, s.pos0,
                s.pos0 + s.q_len, ring->d.n_slots, ring->d.max_pos);
      return AF_ERR_OUT_OF_RANGE;
    }
    if (slot_used[s.slot]) {
      set_error("segment %d: slot %d used by two segments", i, s.slot);
      return AF_ERR_INVALID_ARG;
    }
    slot_used[s.slot] = 1;
    if (ring->owner[s.slot] != s.request_id || ring->len[s.slot] != s.pos0 + s.q_len) {
      set_error("segment %d (request %lld, slot %d, kv_len %d) disagrees with the ring (owner %lld, len %d)", i,
                (long long)s.request_id, s.slot, s.pos0 + s.q_len, (long long)ring->owner[s.slot], ring->len[s.slot]);
      return AF_ERR_INVALID_ARG;
    }
  }
  std::sort(order.begin(), order.end(), [&](int a, int b) { return segs[a].q_start < segs[b].q_start; });
  int next = 0;
  for (int i : order) {
    if (segs[i].q_start != next) {
      set_error("segments must tile rows [0, %d) exactly once (gap or overlap at row %d)", M, next);
      return AF_ERR_INVALID_ARG;
    }
    next += segs[i].q_len;
  }
  if (next != M) {
    set_error("segments cover %d rows, M is %d", next, M);
    return AF_ERR_INVALID_ARG;
  }
  return AF_OK;
}

// Host-built per-call tables (offsets in int32 elements).
struct StepDesc {
  std::vector<int32_t> buf;
  size_t off_segs = 0, off_rows = 0, off_tiles = 0, off_emit = 0;
  int n_tiles = 0, n_multi = 0, n_emit = 0;
};

void build_desc(const af_segment* segs, int n_seg, int M, StepDesc& sd) {
  std::vector<int> emit_idx(n_seg, -1);
  int n_emit = 0;
  for (int i = 0; i < n_seg; ++i)
    if (segs[i].flags & AF_SEG_EMIT) emit_idx[i] = n_emit++;
  // attention work: query tiles of multi-row segments (largest work first, latest tiles first),
  // then the single-row segments, which the decode kernel splits over their keys instead
  std::vector<std::pair<int, int>> tiles;
  std::vector<int> by_len(n_seg);
  std::iota(by_len.begin(), by_len.end(), 0);
  std::stable_sort(by_len.begin(), by_len.end(), [&](int a, int b) {
    const bool ma = segs[a].q_len > 1, mb = segs[b].q_len > 1;
    if (ma != mb) return ma;
    return (int64_t)segs[a].q_len * (segs[a].pos0 + segs[a].q_len) > (int64_t)segs[b].q_len * (segs[b].pos0 + segs[b].q_len);
  });
  sd.n_multi = 0;
  for (int i : by_len) {
    const int nt = (segs[i].q_len + ATTN_BQ - 1) / ATTN_BQ;
    for (int t = nt - 1; t >= 0; --t) tiles.push_back({i, t * ATTN_BQ});
    if (segs[i].q_len > 1) sd.n_multi += nt;
  }
  sd.n_tiles = (int)tiles.size();
  sd.n_emit = n_emit;
  sd.off_segs = 0;
  sd.off_rows = (size_t)n_seg * 8;
  sd.off_tiles = sd.off_rows + (size_t)M * 2;
  sd.off_emit = sd.off_tiles + (size_t)sd.n_tiles * 2;
  sd.buf.assign(sd.off_emit + std::max(n_emit, 1), 0);
  int32_t* b = sd.buf.data();
  for (int i = 0; i < n_seg; ++i) {
    const af_segment& s = segs[i];
    int32_t* ds = b + sd.off_segs + (size_t)i * 8;
    ds[0] = s.q_start;
    ds[1] = s.q_len;
    ds[2] = s.slot;
    ds[3] = s.pos0;
    ds[4] = emit_idx[i];
    for (int r = 0; r < s.q_len; ++r) {
      b[sd.off_rows + 2 * (size_t)(s.q_start + r)] = s.slot;
      b[sd.off_rows + 2 * (size_t)(s.q_start + r) + 1] = s.pos0 + r;
    }
    if (emit_idx[i] >= 0) b[sd.off_emit + emit_idx[i]] = s.q_start + s.q_len - 1;
  }
  for (int t = 0; t < sd.n_tiles; ++t) {
    b[sd.off_tiles + 2 * (size_t)t] = tiles[t].first;
    b[sd.off_tiles + 2 * (size_t)t + 1] = tiles[t].second;
  }
}

// Uploads the descriptor through a rotating set of pinned staging buffers.  Calls on one
// weights object are expected on one stream (the device copy of the descriptor is reused).
af_status upload_desc(af_weights* w, const StepDesc& sd, hipStream_t s) {
  const size_t n = sd.buf.size();
  if (n > w->desc_cap) {
    if (w->desc_dev) {
      AF_HIP(hipDeviceSynchronize());
      dev_free(w, w->desc_dev);
      w->desc_dev = nullptr;
    }
    size_t cap = std::max<size_t>(n, 4096);
    AF_TRY(dev_alloc(w, (void**)&w->desc_dev, cap * 4));
    w->desc_cap = cap;
  }
  StageBuf& sb = w->stage[w->stage_next];
  w->stage_next = (w->stage_next + 1) % 4;
  if (sb.pending) {
    AF_HIP(hipEventSynchronize(sb.done));
    sb.pending = false;
  }
  if (!sb.done) AF_HIP(hipEventCreateWithFlags(&sb.done, hipEventDisableTiming));
  if (n > sb.cap) {
    if (sb.host) (void)hipHostFree(sb.host);
    sb.host = nullptr;
    size_t cap = std::max<size_t>(n, 4096);
    hipError_t e = hipHostMalloc((void**)&sb.host, cap * 4, hipHostMallocDefault);
    if (e != hipSuccess) {
      sb.cap = 0;
      set_error("hipHostMalloc(%zu) failed: %s", cap * 4, hipGetErrorString(e));
      return AF_ERR_OOM;
    }
    sb.cap = cap;
  }
  std::memcpy(sb.host, sd.buf.data(), n * 4);
  AF_HIP(hipMemcpyAsync(w->desc_dev, sb.host, n * 4, hipMemcpyHostToDevice, s));
  AF_HIP(hipEventRecord(sb.done, s));
  sb.pending = true;
  return AF_OK;
}

// Bytes of a GEMM-input activation buffer for `rows` rows of width K (layout per dtype).
size_t act_bytes(const af_weights* w, int rows, bool wide) {
  if (w->d.dtype == AF_BF16) return (size_t)((rows + 31) / 32) * (wide ? w->xs_F : w->xs_D) * w->es;
  return (size_t)rows * (wide ? w->ldF : w->ldD) * w->es;
}

af_status alloc_zeroed(af_weights* w, void** p, size_t bytes) {
  AF_TRY(dev_alloc(w, p, bytes));
  AF_HIP(hipMemset(*p, 0, bytes));
  return AF_OK;
}

af_status ensure_workspace(af_weights* w, int M, int n_emit) {
  const af_model_desc& d = w->d;
  if (M > w->ws_M) {
    AF_HIP(hipDeviceSynchronize());
    dev_free(w, w->xn);
    dev_free(w, w->q);
    dev_free(w, w->attn);
    dev_free(w, w->act);
    w->xn = w->q = w->attn = w->act = nullptr;
    w->ws_M = 0;
    const int cap = std::max(M, 64);
    AF_TRY(alloc_zeroed(w, &w->xn, act_bytes(w, cap, false)));
    AF_TRY(dev_alloc(w, &w->q, (size_t)cap * w->ldD * w->es));
    AF_TRY(alloc_zeroed(w, &w->attn, act_bytes(w, cap, false)));
    AF_TRY(alloc_zeroed(w, &w->act, act_bytes(w, cap, true)));
    w->ws_M = cap;
  }
  if (n_emit > w->ws_emit) {
    AF_HIP(hipDeviceSynchronize());
    dev_free(w, w->emit_norm);
    dev_free(w, w->logits_ws);
    dev_free(w, w->tokens_ws);
    w->emit_norm = nullptr;
    w->logits_ws = nullptr;
    w->tokens_ws = nullptr;
    w->ws_emit = 0;
    const int cap = std::max(n_emit, 16);
    AF_TRY(alloc_zeroed(w, &w->emit_norm, act_bytes(w, cap, false)));
    AF_TRY(dev_alloc(w, (void**)&w->logits_ws, (size_t)cap * d.vocab * 4));
    AF_TRY(dev_alloc(w, (void**)&w->tokens_ws, (size_t)cap * 4));
    w->ws_emit = cap;
  }
  return AF_OK;
}

// Rotary table [pos][j][cos, sin] at angle pos * theta^(-2j/hd), evaluated in double.
af_status ensure_rope(af_weights* w, int max_pos) {
  if (max_pos <= w->rope_cap) return AF_OK;
  const int half = w->d.head_dim / 2;
  std::vector<float> t((size_t)max_pos * half * 2);
  for (int p = 0; p < max_pos; ++p)
    for (int j = 0; j < half; ++j) {
      const double ang = (double)p * std::pow((double)w->d.rope_theta, -2.0 * j / w->d.head_dim);
      t[((size_t)p * half + j) * 2] = (float)std::cos(ang);
      t[((size_t)p * half + j) * 2 + 1] = (float)std::sin(ang);
    }
  AF_HIP(hipDeviceSynchronize());
  dev_free(w, w->rope_cs);
  w->rope_cs = nullptr;
  w->rope_cap = 0;
  AF_TRY(dev_alloc(w, (void**)&w->rope_cs, t.size() * 4));
  AF_HIP(hipMemcpy(w->rope_cs, t.data(), t.size() * 4, hipMemcpyHostToDevice));
  w->rope_cap = max_pos;
  return AF_OK;
}

Ws ws_of(af_weights* w) {
  Ws ws;
  ws.grow = w;
  ws.timing = w;
  ws.xn = w->xn;
  ws.q = w->q;
  ws.attn = w->attn;
  ws.act = w->act;
  ws.emit_norm = w->emit_norm;
  ws.logits = w->logits_ws;
  ws.desc = w->desc_dev;
  ws.rope = w->rope_cs;
  ws.partial = w->partial;
  ws.partial_cap = w->partial_cap;
  return ws;
}

// ---------------------------------------------------------------- timed launches
hipEvent_t take_event(af_weights* w) {
  if (!w->event_pool.empty()) {
    hipEvent_t e = w->event_pool.back();
    w->event_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

template <typename F>
af_status timed(af_weights* w, int cls, hipStream_t s, F&& launch) {
  const bool on = w && (w->timing_mask >> cls) & 1u;
  hipEvent_t a = nullptr, b = nullptr;
  if (on) {
    a = take_event(w);
    b = take_event(w);
    if (!a || !b) {
      set_error("hipEventCreate failed");
      return AF_ERR_DEVICE;
    }
    AF_HIP(hipEventRecord(a, s));
  }
  hipError_t e = launch();
  if (e != hipSuccess) {
    set_error("kernel launch (class %d) failed: %s", cls, hipGetErrorString(e));
    return AF_ERR_DEVICE;
  }
  if (on) {
    AF_HIP(hipEventRecord(b, s));
    w->timed.push_back({cls, a, b});
  }
  return AF_OK;
}

// ---------------------------------------------------------------- steps of Alg. 2
struct DevTables {
  const DevSeg* segs;
  const int32_t* row_sp;
  const int32_t* tiles;
  const int32_t* emit_rows;
  int n_tiles, n_multi, n_emit;
};

DevTables dev_tables(const int32_t* desc, const StepDesc& sd) {
  DevTables t;
  t.segs = (const DevSeg*)(desc + sd.off_segs);
  t.row_sp = desc + sd.off_rows;
  t.tiles = desc + sd.off_tiles;
  t.emit_rows = desc + sd.off_emit;
  t.n_tiles = sd.n_tiles;
  t.n_multi = sd.n_multi;
  t.n_emit = sd.n_emit;
  return t;
}

// A is row-major with stride lda (fp32) or fragment-tiled with block stride astride (bf16).
GemmArgs gemm_args(int dtype, const void* A, int lda, long astride, const void* B, int M, int N, int K, void* out,
                   int ldo) {
  GemmArgs g;
  std::memset(&g, 0, sizeof(g));
  g.A = A;
  g.lda = lda;
  g.astride = astride;
  g.B = B;
  g.M = M;
  g.N = N;
  g.K = K;
  g.Kp = padk(K);
  g.bstride = frag_bstride(g.Kp, dtype);
  g.splits = 1;
  g.out = out;
  g.ldo = ldo;
  return g;
}

// fp32 elements of split-K partial sums a GEMM of this shape needs (0: no split).
size_t split_need(const af_weights* w, int M, int N, int K) {
  if (w->options & AF_OPT_NO_SPLIT_K) return 0;
  const int S = gemm_splits(w->d.dtype, M, N, padk(K));
  return S > 1 ? (size_t)S * M * N : 0;
}

af_status with_splits(af_weights* w, Ws& ws, GemmArgs& g) {
  if (!w || (w->options & AF_OPT_NO_SPLIT_K)) return AF_OK;
  const int S = gemm_splits(w->d.dtype, g.M, g.N, g.Kp);
  if (S <= 1) return AF_OK;
  const size_t need = (size_t)S * g.M * g.N;
  if (need > ws.partial_cap) {
    if (!ws.grow) {
      set_error("split-K partial buffer too small (%zu floats, need %zu)", ws.partial_cap, need);
      return AF_ERR_OUT_OF_RANGE;
    }
    AF_HIP(hipDeviceSynchronize());
    dev_free(w, w->partial);
    w->partial = nullptr;
    w->partial_cap = 0;
    AF_TRY(dev_alloc(w, (void**)&w->partial, need * 4));
    w->partial_cap = need;
    ws.partial = w->partial;
    ws.partial_cap = need;
  }
  g.splits = S;
  g.partial = ws.partial;
  return AF_OK;
}

// l: the weights' layer; rl: the ring layer that holds this layer's keys and values.
af_status step_qkv(af_weights* w, Ws& ws, int l, const void* xn, int ldx, long xs, int M, af_ring* ring, int rl,
                   const DevTables& t, void* q_out, int ldq, hipStream_t s) {
  const af_model_desc& d = w->d;
  GemmArgs g = gemm_args(d.dtype, xn, ldx, xs, w->layers[l].wqkv, M, 3 * d.d_model, d.d_model, q_out, ldq);
  const size_t es = w->es;
  g.ring_k = (char*)ring->kv + ring->offset(rl, 0, 0, 0, 0) * es;
  g.ring_v = (char*)ring->kv + ring->offset(rl, 1, 0, 0, 0) * es;
  g.row_sp = t.row_sp;
  g.rope_cs = ws.rope;
  g.d_model = d.d_model;
  g.head_dim = d.head_dim;
  g.n_heads = d.n_heads;
  g.max_pos = ring->d.max_pos;
  AF_TRY(with_splits(w, ws, g));
  return timed(ws.timing, AF_K_GEMM_QKV, s, [&] { return launch_gemm(d.dtype, EPI_QKV, g, s); });
}

af_status step_attention(af_weights* tw, int dtype, af_ring* ring, int l, const void* q, int ldq, void* o, int ldo,
                         long os, const DevTables& t, hipStream_t s) {
  AttnArgs a;
  std::memset(&a, 0, sizeof(a));
  const size_t es = dtype_size(dtype);
  a.q = q;
  a.o = o;
  a.ring_k = (char*)ring->kv + ring->offset(l, 0, 0, 0, 0) * es;
  a.ring_v = (char*)ring->kv + ring->offset(l, 1, 0, 0, 0) * es;
  a.segs = t.segs;
  a.tiles = t.tiles;
  a.n_multi = t.n_multi;
  a.n_heads = ring->d.n_kv_heads;
  a.max_pos = ring->d.max_pos;
  a.ldq = ldq;
  a.ldo = ldo;
  a.ostride = os;
  a.scale_log2 = (float)(1.4426950408889634 / std::sqrt((double)ring->d.head_dim));
  return timed(tw, AF_K_ATTENTION, s, [&] { return launch_attention(dtype, ring->d.head_dim, a, t.n_tiles, s); });
}

// Residual projections (output and down).  With split-K and a norm gain, the partial sums, the
// residual update and the RMSNorm of the updated rows (gain `norm`, into ws.xn) run as one
// kernel after the GEMM; *normed tells the caller whether that norm was produced.
af_status step_resid_proj(af_weights* w, Ws& ws, int cls, const void* A, int lda, long as, const void* W, int K,
                          void* hidden, int M, const void* norm, bool* normed, hipStream_t s) {
  const af_model_desc& d = w->d;
  GemmArgs g = gemm_args(d.dtype, A, lda, as, W, M, d.d_model, K, hidden, d.d_model);
  g.resid = hidden;
  g.ldr = d.d_model;
  AF_TRY(with_splits(w, ws, g));
  *normed = norm && g.splits > 1;
  if (!*normed) return timed(ws.timing, cls, s, [&] { return launch_gemm(d.dtype, EPI_RESID, g, s); });
  g.partials_only = 1;
  return timed(ws.timing, cls, s, [&] {
    hipError_t e = launch_gemm(d.dtype, EPI_RESID, g, s);
    if (e != hipSuccess) return e;
    return launch_resid_norm(d.dtype, g.partial, g.splits, hidden, d.d_model, norm, ws.xn, w->ldD, w->xs_D, M,
                             d.d_model, d.rms_eps, s);
  });
}

af_status step_o(af_weights* w, Ws& ws, int l, const void* o, int ldo_in, long os, void* hidden, int M, hipStream_t s,
                 const void* norm = nullptr, bool* normed = nullptr) {
  bool dummy;
  return step_resid_proj(w, ws, AF_K_GEMM_O, o, ldo_in, os, w->layers[l].wo, w->d.d_model, hidden, M, norm,
                         normed ? normed : &dummy, s);
}

af_status step_gate_up(af_weights* w, Ws& ws, int l, const void* xn, int ldx, long xs, void* act, int ld_act,
                       long act_os, int M, hipStream_t s) {
  const af_model_desc& d = w->d;
  GemmArgs g = gemm_args(d.dtype, xn, ldx, xs, w->layers[l].wgu, M, 2 * d.d_ff, d.d_model, act, ld_act);
  g.ostride = act_os;
  AF_TRY(with_splits(w, ws, g));
  return timed(ws.timing, AF_K_GEMM_GATEUP, s, [&] { return launch_gemm(d.dtype, EPI_SWIGLU, g, s); });
}

af_status step_down(af_weights* w, Ws& ws, int l, const void* act, int ld_act, long as, void* hidden, int M,
                    hipStream_t s, const void* norm = nullptr, bool* normed = nullptr) {
  bool dummy;
  return step_resid_proj(w, ws, AF_K_GEMM_DOWN, act, ld_act, as, w->layers[l].wdown, w->d.d_ff, hidden, M, norm,
                         normed ? normed : &dummy, s);
}

af_status step_norm(af_weights* w, af_weights* tw, const void* x, int ldx, const int32_t* rows, const void* g,
                    void* y, int ldy, long ys, int n_rows, hipStream_t s) {
  const af_model_desc& d = w->d;
  return timed(tw, AF_K_RMSNORM, s, [&] {
    return launch_rmsnorm(d.dtype, x, ldx, rows, g, y, ldy, ys, n_rows, d.d_model, d.rms_eps, s);
  });
}

// One decoder layer (Alg. 2).  xn_ready: the previous layer's down projection already wrote
// this layer's attention-normed rows into ws.xn.  next_norm: the next layer's attention-norm
// gain, which this layer's down projection applies when it can (*next_ready then says so).
// Layer l of the weights; its keys and values live in ring layer rl.
af_status layer_forward(af_weights* w, Ws& ws, int l, void* hidden, int M, af_ring* ring, int rl, const DevTables& t,
                        hipStream_t s, bool xn_ready = false, const void* next_norm = nullptr,
                        bool* next_ready = nullptr) {
  const Layer& L = w->layers[l];
  const int D = w->d.d_model, ldD = w->ldD, ldF = w->ldF;
  const long xD = w->xs_D, xF = w->xs_F;  // 0 (row-major) for fp32
  if (!xn_ready) AF_TRY(step_norm(w, ws.timing, hidden, D, nullptr, L.attn_norm, ws.xn, ldD, xD, M, s));
  AF_TRY(step_qkv(w, ws, l, ws.xn, ldD, xD, M, ring, rl, t, ws.q, ldD, s));
  AF_TRY(step_attention(ws.timing, w->d.dtype, ring, rl, ws.q, ldD, ws.attn, ldD, xD, t, s));
  // InPlaceKVShift: no device work; the slot rotation lives in the ring bookkeeping.
  bool mlp_normed = false;
  AF_TRY(step_o(w, ws, l, ws.attn, ldD, xD, hidden, M, s, L.mlp_norm, &mlp_normed));
  if (!mlp_normed) AF_TRY(step_norm(w, ws.timing, hidden, D, nullptr, L.mlp_norm, ws.xn, ldD, xD, M, s));
  AF_TRY(step_gate_up(w, ws, l, ws.xn, ldD, xD, ws.act, ldF, xF, M, s));
  bool dummy;
  AF_TRY(step_down(w, ws, l, ws.act, ldF, xF, hidden, M, s, next_norm, next_ready ? next_ready : &dummy));
  return AF_OK;
}

af_status lm_head(af_weights* w, Ws& ws, const void* hidden, const DevTables& t, float* out_logits,
                  int32_t* out_tokens, hipStream_t s) {
  const af_model_desc& d = w->d;
  if (t.n_emit == 0 || (!out_logits && !out_tokens)) return AF_OK;
  AF_TRY(step_norm(w, ws.timing, hidden, d.d_model, t.emit_rows, w->final_norm, ws.emit_norm, w->ldD, w->xs_D,
                   t.n_emit, s));
  float* logits = out_logits ? out_logits : ws.logits;
  GemmArgs g = gemm_args(d.dtype, ws.emit_norm, w->ldD, w->xs_D, w->lm_head, t.n_emit, d.vocab, d.d_model, logits,
                         d.vocab);
  AF_TRY(with_splits(w, ws, g));
  AF_TRY(timed(ws.timing, AF_K_LM_HEAD, s, [&] { return launch_gemm(d.dtype, EPI_STORE_F32, g, s); }));
  if (out_tokens)
    AF_TRY(timed(ws.timing, AF_K_ARGMAX, s, [&] { return launch_argmax(logits, t.n_emit, d.vocab, out_tokens, s); }));
  return AF_OK;
}

af_status prepare_step(af_weights* w, af_ring* ring, const af_segment* segs, int n_seg, int M, int min_layers,
                       StepDesc& sd, hipStream_t s) {
  AF_TRY(check_ring_matches(w, ring, min_layers));
  AF_TRY(check_segments(ring, segs, n_seg, M));
  build_desc(segs, n_seg, M, sd);
  AF_TRY(ensure_workspace(w, M, sd.n_emit));
  AF_TRY(ensure_rope(w, ring->d.max_pos));
  AF_TRY(upload_desc(w, sd, s));
  return AF_OK;
}

// The whole step (Alg. 1 Embed .. ArgMax) on a prepared workspace and uploaded tables.
af_status forward_steps(af_weights* w, Ws& ws, const DevTables& t, const int32_t* token_ids, const void* embeds,
                        int M, af_ring* ring, void* out_hidden, float* out_logits, int32_t* out_tokens,
                        hipStream_t s) {
  const af_model_desc& d = w->d;
  AF_TRY(timed(ws.timing, AF_K_EMBED, s, [&] {
    return launch_embed(d.dtype, token_ids, w->embed, d.vocab, embeds, out_hidden, M, d.d_model, w->dev_err, s);
  }));
  bool xn_ready = false;
  for (int l = 0; l < d.n_layers; ++l) {
    const void* next = l + 1 < d.n_layers ? w->layers[l + 1].attn_norm : nullptr;
    bool next_ready = false;
    AF_TRY(layer_forward(w, ws, l, out_hidden, M, ring, l, t, s, xn_ready, next, &next_ready));
    xn_ready = next_ready;
  }
  return lm_head(w, ws, out_hidden, t, out_logits, out_tokens, s);
}

af_status check_forward_args(const af_weights* w, const int32_t* token_ids, const void* out_hidden,
                             const af_ring* ring) {
  if (!w || !token_ids || !out_hidden) {
    set_error("af_packed_forward: weights, token_ids and out_hidden must be non-NULL");
    return AF_ERR_INVALID_ARG;
  }
  if (ring && ring->d.n_layers != w->d.n_layers) {
    set_error("af_packed_forward: ring has %d layers, model %d", ring->d.n_layers, w->d.n_layers);
    return AF_ERR_INVALID_ARG;
  }
  return AF_OK;
}

}  // namespace

// ================================================================ weights
extern "C" int32_t af_weights_tensor_count(int32_t n_layers) { return 3 + 9 * n_layers; }

extern "C" af_status af_weights_destroy(af_weights* w) {
  clear_error();
  if (!w) return AF_OK;
  (void)hipDeviceSynchronize();
  for (void* p : w->allocs) (void)hipFree(p);
  for (auto& sb : w->stage) {
    if (sb.host) (void)hipHostFree(sb.host);
    if (sb.done) (void)hipEventDestroy(sb.done);
  }
  for (auto& t : w->timed) {
    (void)hipEventDestroy(t.start);
    (void)hipEventDestroy(t.stop);
  }
  for (hipEvent_t e : w->event_pool) (void)hipEventDestroy(e);
  delete w;
  return AF_OK;
}

extern "C" af_status af_weights_create(const af_model_desc* desc, const void* const* tensors, int32_t n_tensors,
                                       void* hip_stream, af_weights** out) {
  clear_error();
  if (!desc || !tensors || !out) {
    set_error("af_weights_create: desc, tensors and out must be non-NULL");
    return AF_ERR_INVALID_ARG;
  }
  *out = nullptr;
  AF_TRY(check_model_desc(*desc));
  const af_model_desc& d = *desc;
  if (n_tensors != af_weights_tensor_count(d.n_layers)) {
    set_error("af_weights_create: expected %d tensors, got %d", af_weights_tensor_count(d.n_layers), n_tensors);
    return AF_ERR_INVALID_ARG;
  }
  for (int i = 0; i < n_tensors; ++i)
    if (!tensors[i]) {
      set_error("af_weights_create: tensor %d is NULL", i);
      return AF_ERR_INVALID_ARG;
    }
  af_weights* w = new (std::nothrow) af_weights();
  if (!w) {
    set_error("af_weights_create: host allocation failed");
    return AF_ERR_OOM;
  }
  w->d = d;
  w->es = dtype_size(d.dtype);
  w->ldD = d.d_model + STRIDE_PAD_BYTES / (int)w->es;
  w->ldF = d.d_ff + STRIDE_PAD_BYTES / (int)w->es;
  if (d.dtype == AF_BF16) {
    w->xs_D = frag_astride(padk(d.d_model));
    w->xs_F = frag_astride(padk(d.d_ff));
  }
  hipStream_t s = (hipStream_t)hip_stream;
  const size_t es = w->es;
  const int D = d.d_model, F = d.d_ff, V = d.vocab, hd = d.head_dim;
  auto fail = [&](af_status st) {
    af_weights_destroy(w);
    return st;
  };
  auto copy_new = [&](void** dst, const void* src, size_t bytes) -> af_status {
    AF_TRY(dev_alloc(w, dst, bytes));
    AF_HIP(hipMemcpyAsync(*dst, src, bytes, hipMemcpyDeviceToDevice, s));
    return AF_OK;
  };
  af_status st;
  if ((st = copy_new(&w->embed, tensors[0], (size_t)V * D * es)) != AF_OK) return fail(st);
  if ((st = copy_new(&w->final_norm, tensors[1], (size_t)D * es)) != AF_OK) return fail(st);

  // Row maps of the fused projections (source tensor, source row) per output row.  Every
  // 16-row block holds 8 a-rows and then their 8 partners, so the GEMM epilogue finds a
  // partner one lane away.  QKV: for each of q, k, v and each head, block p holds dims
  // [8p, 8p + 8) and [hd/2 + 8p, hd/2 + 8p + 8) (the rotary pairs).
  std::vector<int32_t> qkv_map((size_t)3 * D * 2), gu_map((size_t)2 * F * 2);
  for (int c = 0; c < 3 * D; ++c) {
    const int region = c / D, cr = c % D, h = cr / hd, jj = cr % hd;
    const int dim = (jj >> 4) * 8 + (jj & 7) + ((jj & 8) ? hd / 2 : 0);
    qkv_map[2 * c] = region;
    qkv_map[2 * c + 1] = h * hd + dim;
  }
  // gate/up: block p holds gate rows [8p, 8p + 8) and up rows [8p, 8p + 8).
  for (int c = 0; c < 2 * F; ++c) {
    gu_map[2 * c] = (c & 8) ? 1 : 0;
    gu_map[2 * c + 1] = (c >> 4) * 8 + (c & 7);
  }
  // device array of source pointers: per layer [wq, wk, wv, w_gate, w_up, wo, w_down, -], then lm_head
  const size_t n_ptr = (size_t)d.n_layers * 8 + 8;
  std::vector<const void*> srcs(n_ptr, nullptr);
  for (int l = 0; l < d.n_layers; ++l) {
    const void* const* t = tensors + 3 + 9 * l;
    srcs[8 * l + 0] = t[1];
    srcs[8 * l + 1] = t[2];
    srcs[8 * l + 2] = t[3];
    srcs[8 * l + 3] = t[6];
    srcs[8 * l + 4] = t[7];
    srcs[8 * l + 5] = t[4];
    srcs[8 * l + 6] = t[8];
  }
  srcs[(size_t)d.n_layers * 8] = tensors[2];
  int32_t *qkv_map_d = nullptr, *gu_map_d = nullptr;
  const void** srcs_d = nullptr;
  if ((st = dev_alloc(w, (void**)&qkv_map_d, qkv_map.size() * 4)) != AF_OK) return fail(st);
  if ((st = dev_alloc(w, (void**)&gu_map_d, gu_map.size() * 4)) != AF_OK) return fail(st);
  if ((st = dev_alloc(w, (void**)&srcs_d, n_ptr * sizeof(void*))) != AF_OK) return fail(st);
  hipError_t he = hipMemcpy(qkv_map_d, qkv_map.data(), qkv_map.size() * 4, hipMemcpyHostToDevice);
  if (he == hipSuccess) he = hipMemcpy(gu_map_d, gu_map.data(), gu_map.size() * 4, hipMemcpyHostToDevice);
  if (he == hipSuccess) he = hipMemcpy(srcs_d, srcs.data(), n_ptr * sizeof(void*), hipMemcpyHostToDevice);
  if (he != hipSuccess) {
    set_error("af_weights_create: map upload failed: %s", hipGetErrorString(he));
    return fail(AF_ERR_DEVICE);
  }
  const int Dp = padk(D), Fp = padk(F);
  auto pack = [&](void** dst, const void* const* src_d, const int32_t* map, int N, int K, int Kp) -> af_status {
    const long bs = frag_bstride(Kp, d.dtype);
    const int nc = frag_ncols(d.dtype);
    AF_TRY(dev_alloc(w, dst, (size_t)((N + nc - 1) / nc) * bs * es));
    AF_HIP(launch_frag_pack(d.dtype, *dst, bs, src_d, map, N, K, Kp, s));
    return AF_OK;
  };
  if ((st = pack(&w->lm_head, srcs_d + (size_t)d.n_layers * 8, nullptr, V, D, Dp)) != AF_OK) return fail(st);
  w->layers.resize(d.n_layers);
  for (int l = 0; l < d.n_layers; ++l) {
    const void* const* t = tensors + 3 + 9 * l;
    Layer& L = w->layers[l];
    const void* const* sl = srcs_d + 8 * (size_t)l;
    if ((st = copy_new(&L.attn_norm, t[0], (size_t)D * es)) != AF_OK) return fail(st);
    if ((st = copy_new(&L.mlp_norm, t[5], (size_t)D * es)) != AF_OK) return fail(st);
    if ((st = pack(&L.wqkv, sl, qkv_map_d, 3 * D, D, Dp)) != AF_OK) return fail(st);
    if ((st = pack(&L.wgu, sl + 3, gu_map_d, 2 * F, D, Dp)) != AF_OK) return fail(st);
    if ((st = pack(&L.wo, sl + 5, nullptr, D, D, Dp)) != AF_OK) return fail(st);
    if ((st = pack(&L.wdown, sl + 6, nullptr, D, F, Fp)) != AF_OK) return fail(st);
  }
  if ((st = dev_alloc(w, (void**)&w->dev_err, 64)) != AF_OK) return fail(st);
  he = hipMemsetAsync(w->dev_err, 0, 64, s);
  if (he == hipSuccess) he = hipStreamSynchronize(s);
  if (he != hipSuccess) {
    set_error("af_weights_create: %s", hipGetErrorString(he));
    return fail(AF_ERR_DEVICE);
  }
  dev_free(w, qkv_map_d);
  dev_free(w, gu_map_d);
  dev_free(w, (void*)srcs_d);
  *out = w;
  return AF_OK;
}

extern "C" af_status af_weights_device_errors(af_weights* w, void* hip_stream, int32_t* count) {
  clear_error();
  if (!w || !count) {
    set_error("af_weights_device_errors: NULL argument");
    return AF_ERR_INVALID_ARG;
  }
  hipStream_t s = (hipStream_t)hip_stream;
  AF_HIP(hipStreamSynchronize(s));
  AF_HIP(hipMemcpy(count, w->dev_err, 4, hipMemcpyDeviceToHost));
  AF_HIP(hipMemset(w->dev_err, 0, 4));
  return AF_OK;
}

// ================================================================ forward
extern "C" af_status af_packed_forward(af_weights* w, const int32_t* token_ids, const void* embeds, int32_t M,
                                       const af_segment* segs, int32_t n_seg, af_ring* ring, void* out_hidden,
                                       float* out_logits, int32_t* out_tokens, void* hip_stream) {
  clear_error();
  AF_TRY(check_forward_args(w, token_ids, out_hidden, ring));
  hipStream_t s = (hipStream_t)hip_stream;
  StepDesc sd;
  AF_TRY(prepare_step(w, ring, segs, n_seg, M, w->d.n_layers, sd, s));
  Ws ws = ws_of(w);
  return forward_steps(w, ws, dev_tables(ws.desc, sd), token_ids, embeds, M, ring, out_hidden, out_logits,
                       out_tokens, s);
}

extern "C" af_status af_packed_layer_forward(af_weights* w, int32_t layer, void* hidden_inout, int32_t M,
                                             const af_segment* segs, int32_t n_seg, af_ring* ring, void* hip_stream) {
  clear_error();
  return af_packed_layer_forward_kv(w, layer, hidden_inout, M, segs, n_seg, ring, layer, hip_stream);
}

extern "C" af_status af_packed_layer_forward_kv(af_weights* w, int32_t layer, void* hidden_inout, int32_t M,
                                                const af_segment* segs, int32_t n_seg, af_ring* ring,
                                                int32_t ring_layer, void* hip_stream) {
  clear_error();
  if (!w || !hidden_inout) {
    set_error("af_packed_layer_forward: weights and hidden must be non-NULL");
    return AF_ERR_INVALID_ARG;
  }
  if (layer < 0 || layer >= w->d.n_layers) {
    set_error("af_packed_layer_forward: layer %d outside [0, %d)", layer, w->d.n_layers);
    return AF_ERR_OUT_OF_RANGE;
  }
  if (ring_layer < 0) {
    set_error("af_packed_layer_forward: ring layer %d is negative", ring_layer);
    return AF_ERR_OUT_OF_RANGE;
  }
  hipStream_t s = (hipStream_t)hip_stream;
  StepDesc sd;
  AF_TRY(prepare_step(w, ring, segs, n_seg, M, ring_layer + 1, sd, s));
  Ws ws = ws_of(w);
  return layer_forward(w, ws, layer, hidden_inout, M, ring, ring_layer, dev_tables(ws.desc, sd), s);
}

// ================================================================ forward in a caller-free buffer
// The step of af_packed_forward with every device workspace carved from one fixed buffer: no
// device or pinned-host allocation.  Layout (256-byte aligned regions): rotary table, step
// tables, xn, attn, act, q, emit_norm, fp32 logits (only when tokens are wanted without
// logits), split-K partials (the largest any GEMM of the step needs).  The rotary table is
// uploaded only when *rope says the buffer does not already hold it.
af_status af::packed_forward_in_buffer(af_weights* w, const int32_t* token_ids, const void* embeds, int32_t M,
                                       const af_segment* segs, int32_t n_seg, af_ring* ring, void* out_hidden,
                                       float* out_logits, int32_t* out_tokens, hipStream_t s, void* buf,
                                       size_t buf_bytes, BufferRope* rope) {
  AF_TRY(check_forward_args(w, token_ids, out_hidden, ring));
  AF_TRY(check_ring_matches(w, ring, w->d.n_layers));
  AF_TRY(check_segments(ring, segs, n_seg, M));
  const af_model_desc& d = w->d;
  StepDesc sd;
  build_desc(segs, n_seg, M, sd);
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += (bytes + 255) / 256 * 256;
    return o;
  };
  const int half = d.head_dim / 2, max_pos = ring->d.max_pos;
  const size_t o_rope = take((size_t)max_pos * half * 2 * 4);
  const size_t o_desc = take(sd.buf.size() * 4);
  const size_t o_xn = take(act_bytes(w, M, false));
  const size_t o_attn = take(act_bytes(w, M, false));
  const size_t o_act = take(act_bytes(w, M, true));
  const size_t o_q = take((size_t)M * w->ldD * w->es);
  const int n_emit = sd.n_emit;
  const size_t o_emit = take(act_bytes(w, std::max(n_emit, 1), false));
  const bool head = n_emit > 0 && (out_logits || out_tokens);
  const size_t o_logits = take(head && !out_logits ? (size_t)n_emit * d.vocab * 4 : 0);
  size_t part = std::max({split_need(w, M, 3 * d.d_model, d.d_model), split_need(w, M, d.d_model, d.d_model),
                          split_need(w, M, 2 * d.d_ff, d.d_model), split_need(w, M, d.d_model, d.d_ff)});
  if (head) part = std::max(part, split_need(w, n_emit, d.vocab, d.d_model));
  const size_t o_part = take(part * 4);
  if (off > buf_bytes) {
    set_error("af_packed_forward_noalloc: this step needs %zu bytes of scratch (M = %d, d_model %d, d_ff %d, "
              "ring max_pos %d, %d emitting rows); the library holds %zu",
              off, M, d.d_model, d.d_ff, max_pos, n_emit, buf_bytes);
    return AF_ERR_OUT_OF_RANGE;
  }
  char* base = (char*)buf;
  if (!(rope->theta == d.rope_theta && rope->head_dim == d.head_dim && rope->rows >= max_pos)) {
    std::vector<float> t((size_t)max_pos * half * 2);
    for (int p = 0; p < max_pos; ++p)
      for (int j = 0; j < half; ++j) {
        const double ang = (double)p * std::pow((double)d.rope_theta, -2.0 * j / d.head_dim);
        t[((size_t)p * half + j) * 2] = (float)std::cos(ang);
        t[((size_t)p * half + j) * 2 + 1] = (float)std::sin(ang);
      }
    rope->rows = 0;
    AF_HIP(hipMemcpyAsync(base + o_rope, t.data(), t.size() * 4, hipMemcpyHostToDevice, s));
  }
  rope->theta = d.rope_theta;
  rope->head_dim = d.head_dim;
  rope->rows = max_pos;  // what lies past this call's table may be overwritten by its other regions
  AF_HIP(hipMemcpyAsync(base + o_desc, sd.buf.data(), sd.buf.size() * 4, hipMemcpyHostToDevice, s));
  Ws ws;
  ws.xn = base + o_xn;
  ws.attn = base + o_attn;
  ws.act = base + o_act;
  ws.q = base + o_q;
  ws.emit_norm = base + o_emit;
  ws.logits = (float*)(base + o_logits);
  ws.desc = (int32_t*)(base + o_desc);
  ws.rope = (const float*)(base + o_rope);
  ws.partial = part ? (float*)(base + o_part) : nullptr;
  ws.partial_cap = part;
  if (d.dtype == AF_BF16) {
    // the fragment-tiled GEMM inputs read k up to the padded K: those columns must be zero
    auto zero_pad = [&](void* p, int rows, int K, long xs) -> af_status {
      const int Kp = padk(K);
      if (Kp == K) return AF_OK;
      const size_t head_bytes = (size_t)(K / 16) * 512 * 2, pad_bytes = (size_t)((Kp - K) / 16) * 512 * 2;
      AF_HIP(launch_zero_runs((char*)p + head_bytes, (rows + 31) / 32, (size_t)xs * 2, pad_bytes, s));
      return AF_OK;
    };
    AF_TRY(zero_pad(ws.xn, M, d.d_model, w->xs_D));
    AF_TRY(zero_pad(ws.attn, M, d.d_model, w->xs_D));
    AF_TRY(zero_pad(ws.act, M, d.d_ff, w->xs_F));
    AF_TRY(zero_pad(ws.emit_norm, std::max(n_emit, 1), d.d_model, w->xs_D));
  }
  return forward_steps(w, ws, dev_tables(ws.desc, sd), token_ids, embeds, M, ring, out_hidden, out_logits,
                       out_tokens, s);
}

// ================================================================ single steps
extern "C" af_status af_op_embed(af_weights* w, const int32_t* token_ids, const void* embeds, int32_t M, void* out,
                                 void* hip_stream) {
  clear_error();
  if (!w || !token_ids || !out || M <= 0) {
    set_error("af_op_embed: bad argument");
    return AF_ERR_INVALID_ARG;
  }
  hipStream_t s = (hipStream_t)hip_stream;
  return timed(w, AF_K_EMBED, s, [&] {
    return launch_embed(w->d.dtype, token_ids, w->embed, w->d.vocab, embeds, out, M, w->d.d_model, w->dev_err, s);
  });
}

extern "C" af_status af_op_rmsnorm(int32_t dtype, const void* x, const void* g, void* y, int32_t M, int32_t D,
                                   float eps, void* hip_stream) {
  clear_error();
  if ((dtype != AF_BF16 && dtype != AF_F32) || !x || !g || !y || M <= 0 || D <= 0) {
    set_error("af_op_rmsnorm: bad argument");
    return AF_ERR_INVALID_ARG;
  }
  AF_HIP(launch_rmsnorm(dtype, x, D, nullptr, g, y, D, 0, M, D, eps, (hipStream_t)hip_stream));
  return AF_OK;
}

extern "C" af_status af_op_linear(int32_t dtype, const void* x, const void* wt, void* y, int32_t M, int32_t N, int32_t K,
                                  void* hip_stream) {
  clear_error();
  const int vec = dtype == AF_BF16 ? 8 : 4;
  if ((dtype != AF_BF16 && dtype != AF_F32) || !x || !wt || !y || M <= 0 || N <= 0 || K <= 0) {
    set_error("af_op_linear: bad argument");
    return AF_ERR_INVALID_ARG;
  }
  if (K % vec != 0 || N % 16 != 0) {
    set_error("af_op_linear: need K %% %d == 0 and N %% 16 == 0", vec);
    return AF_ERR_UNSUPPORTED;
  }
  // the caller's weight is row-major [N, K]: fragment-tile a private copy (synchronous)
  hipStream_t s = (hipStream_t)hip_stream;
  const int Kp = padk(K), nc = frag_ncols(dtype);
  void *wf = nullptr, *xf = nullptr;
  const void** src_d = nullptr;
  const long bs = frag_bstride(Kp, dtype);
  const long xs = dtype == AF_BF16 ? frag_astride(Kp) : 0;  // bf16 reads fragment-tiled activations
  AF_HIP(hipMalloc(&wf, (size_t)((N + nc - 1) / nc) * bs * dtype_size(dtype)));
  hipError_t e = hipMalloc((void**)&src_d, sizeof(void*));
  if (e == hipSuccess) e = hipMemcpy(src_d, &wt, sizeof(void*), hipMemcpyHostToDevice);
  if (e == hipSuccess) e = launch_frag_pack(dtype, wf, bs, src_d, nullptr, N, K, Kp, s);
  if (e == hipSuccess && xs) {
    e = hipMalloc(&xf, (size_t)((M + 31) / 32) * xs * 2);
    if (e == hipSuccess) e = launch_to_frag(dtype, x, K, M, K, Kp, xf, xs, s);
  }
  float* part = nullptr;
  if (e == hipSuccess) {
    GemmArgs g = gemm_args(dtype, xs ? xf : x, K, xs, wf, M, N, K, y, N);
    g.splits = gemm_splits(dtype, M, N, Kp);  // the split the model path would use for this shape
    if (g.splits > 1) {
      e = hipMalloc((void**)&part, (size_t)g.splits * M * N * 4);
      g.partial = part;
    }
    if (e == hipSuccess) e = launch_gemm(dtype, EPI_STORE, g, s);
  }
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  (void)hipFree(wf);
  if (xf) (void)hipFree(xf);
  if (part) (void)hipFree(part);
  if (src_d) (void)hipFree(src_d);
  if (e != hipSuccess) {
    set_error("af_op_linear: %s", hipGetErrorString(e));
    return AF_ERR_DEVICE;
  }
  return AF_OK;
}

namespace {
// The single-step entry points take row-major activations.  For bf16 the projection GEMMs read
// fragment-tiled ones: copy the input into the workspace buffer `dst` (stride xs) first.
af_status stage_input(af_weights* w, const void*& x, int K, int M, void* dst, long xs, hipStream_t s) {
  if (!xs) return AF_OK;
  AF_HIP(launch_to_frag(w->d.dtype, x, K, M, K, padk(K), dst, xs, s));
  x = dst;
  return AF_OK;
}
}  // namespace

extern "C" af_status af_op_qkv_rope_write(af_weights* w, int32_t layer, const void* xn, int32_t M,
                                          const af_segment* segs, int32_t n_seg, af_ring* ring, void* q_out,
                                          void* hip_stream) {
  clear_error();
  if (!w || !xn || !q_out || layer < 0 || layer >= w->d.n_layers) {
    set_error("af_op_qkv_rope_write: bad argument");
    return AF_ERR_INVALID_ARG;
  }
  hipStream_t s = (hipStream_t)hip_stream;
  StepDesc sd;
  AF_TRY(prepare_step(w, ring, segs, n_seg, M, layer + 1, sd, s));
  AF_TRY(stage_input(w, xn, w->d.d_model, M, w->xn, w->xs_D, s));
  Ws ws = ws_of(w);
  return step_qkv(w, ws, layer, xn, w->d.d_model, w->xs_D, M, ring, layer, dev_tables(ws.desc, sd), q_out,
                  w->d.d_model, s);
}

extern "C" af_status af_op_attention(af_ring* ring, int32_t layer, const void* q, int32_t M, const af_segment* segs,
                                     int32_t n_seg, void* o, void* hip_stream) {
  clear_error();
  if (!ring || !ring->kv || !q || !o || layer < 0 || layer >= ring->d.n_layers) {
    set_error("af_op_attention: bad argument");
    return AF_ERR_INVALID_ARG;
  }
  AF_TRY(check_segments(ring, segs, n_seg, M));
  StepDesc sd;
  build_desc(segs, n_seg, M, sd);
  hipStream_t s = (hipStream_t)hip_stream;
  // standalone call: private descriptor copy, synchronous
  int32_t* dd = nullptr;
  AF_HIP(hipMalloc(&dd, sd.buf.size() * 4));
  hipError_t e = hipMemcpy(dd, sd.buf.data(), sd.buf.size() * 4, hipMemcpyHostToDevice);
  af_status st = AF_OK;
  if (e == hipSuccess) {
    DevTables t;
    t.segs = (const DevSeg*)(dd + sd.off_segs);
    t.row_sp = dd + sd.off_rows;
    t.tiles = dd + sd.off_tiles;
    t.emit_rows = dd + sd.off_emit;
    t.n_tiles = sd.n_tiles;
    t.n_multi = sd.n_multi;
    t.n_emit = sd.n_emit;
    const int ld = ring->d.n_kv_heads * ring->d.head_dim;
    st = step_attention(nullptr, ring->d.dtype, ring, layer, q, ld, o, ld, 0, t, s);
    if (st == AF_OK) e = hipStreamSynchronize(s);
  }
  (void)hipFree(dd);
  if (e != hipSuccess) {
    set_error("af_op_attention: %s", hipGetErrorString(e));
    return AF_ERR_DEVICE;
  }
  return st;
}

extern "C" af_status af_op_o_proj_residual(af_weights* w, int32_t layer, const void* o, void* hidden, int32_t M,
                                           void* hip_stream) {
  clear_error();
  if (!w || !o || !hidden || M <= 0 || layer < 0 || layer >= w->d.n_layers) {
    set_error("af_op_o_proj_residual: bad argument");
    return AF_ERR_INVALID_ARG;
  }
  hipStream_t s = (hipStream_t)hip_stream;
  AF_TRY(ensure_workspace(w, M, 0));
  AF_TRY(stage_input(w, o, w->d.d_model, M, w->attn, w->xs_D, s));
  Ws ws = ws_of(w);
  return step_o(w, ws, layer, o, w->d.d_model, w->xs_D, hidden, M, s);
}

extern "C" af_status af_op_gate_up_swiglu(af_weights* w, int32_t layer, const void* xn, void* act, int32_t M,
                                          void* hip_stream) {
  clear_error();
  if (!w || !xn || !act || M <= 0 || layer < 0 || layer >= w->d.n_layers) {
    set_error("af_op_gate_up_swiglu: bad argument");
    return AF_ERR_INVALID_ARG;
  }
  hipStream_t s = (hipStream_t)hip_stream;
  AF_TRY(ensure_workspace(w, M, 0));
  AF_TRY(stage_input(w, xn, w->d.d_model, M, w->xn, w->xs_D, s));
  Ws ws = ws_of(w);
  return step_gate_up(w, ws, layer, xn, w->d.d_model, w->xs_D, act, w->d.d_ff, 0, M, s);
}

extern "C" af_status af_op_down_residual(af_weights* w, int32_t layer, const void* act, void* hidden, int32_t M,
                                         void* hip_stream) {
  clear_error();
  if (!w || !act || !hidden || M <= 0 || layer < 0 || layer >= w->d.n_layers) {
    set_error("af_op_down_residual: bad argument");
    return AF_ERR_INVALID_ARG;
  }
  hipStream_t s = (hipStream_t)hip_stream;
  AF_TRY(ensure_workspace(w, M, 0));
  AF_TRY(stage_input(w, act, w->d.d_ff, M, w->act, w->xs_F, s));
  Ws ws = ws_of(w);
  return step_down(w, ws, layer, act, w->d.d_ff, w->xs_F, hidden, M, s);
}

extern "C" af_status af_op_lm_head_argmax(af_weights* w, const void* hidden, int32_t M, const af_segment* segs,
                                          int32_t n_seg, float* out_logits, int32_t* out_tokens, void* hip_stream) {
  clear_error();
  if (!w || !hidden || M <= 0 || !segs || n_seg <= 0 || n_seg > MAX_SEGMENTS) {
    set_error("af_op_lm_head_argmax: bad argument");
    return AF_ERR_INVALID_ARG;
  }
  for (int i = 0; i < n_seg; ++i)
    if (segs[i].q_len <= 0 || segs[i].q_start < 0 || (int64_t)segs[i].q_start + segs[i].q_len > M) {
      set_error("af_op_lm_head_argmax: segment %d outside [0, %d)", i, M);
      return AF_ERR_INVALID_ARG;
    }
  hipStream_t s = (hipStream_t)hip_stream;
  StepDesc sd;
  build_desc(segs, n_seg, M, sd);
  AF_TRY(ensure_workspace(w, M, sd.n_emit));
  AF_TRY(upload_desc(w, sd, s));
  Ws ws = ws_of(w);
  return lm_head(w, ws, hidden, dev_tables(ws.desc, sd), out_logits, out_tokens, s);
}

extern "C" af_status af_weights_set_options(af_weights* w, uint32_t flags) {
  clear_error();
  if (!w || (flags & ~AF_OPT_NO_SPLIT_K)) {
    set_error("af_weights_set_options: bad argument");
    return AF_ERR_INVALID_ARG;
  }
  w->options = flags;
  return AF_OK;
}

// ================================================================ timing
extern "C" af_status af_timing_enable(af_weights* w, uint32_t mask) {
  clear_error();
  if (!w) {
    set_error("af_timing_enable: NULL weights");
    return AF_ERR_INVALID_ARG;
  }
  AF_HIP(hipDeviceSynchronize());
  for (auto& t : w->timed) {
    w->event_pool.push_back(t.start);
    w->event_pool.push_back(t.stop);
  }
  w->timed.clear();
  w->timing_mask = mask;
  return AF_OK;
}

extern "C" af_status af_timing_read(af_weights* w, double* total_ms, int64_t* launches) {
  clear_error();
  if (!w) {
    set_error("af_timing_read: NULL weights");
    return AF_ERR_INVALID_ARG;
  }
  std::vector<double> ms(AF_K_COUNT, 0.0);
  std::vector<int64_t> n(AF_K_COUNT, 0);
  for (auto& t : w->timed) {
    AF_HIP(hipEventSynchronize(t.stop));
    float f = 0.f;
    AF_HIP(hipEventElapsedTime(&f, t.start, t.stop));
    ms[t.cls] += f;
    n[t.cls] += 1;
  }
  if (total_ms) std::copy(ms.begin(), ms.end(), total_ms);
  if (launches) std::copy(n.begin(), n.end(), launches);
  return AF_OK;
}
