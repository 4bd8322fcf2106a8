// Unified KV Ring Buffer (Sec. 3.3): device storage plus the host-side slot rotation that
// replaces the paper's InPlaceKVShift copy.  The bookkeeping is plain integer state and
// never touches the device, so it also runs on machines without a GPU (n_layers == 0).
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>

#include "af_internal.h"

namespace af {

static thread_local char g_err[1024] = "";

void set_error(const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}
void clear_error() { g_err[0] = 0; }
const char* last_error() { return g_err; }

}  // namespace af

using namespace af;

extern "C" const char* af_last_error(void) { return af::last_error(); }

extern "C" af_status af_ring_create(const af_ring_desc* desc, void* hip_stream, af_ring** out) {
  clear_error();
  if (!desc || !out) {
    set_error("af_ring_create: desc and out must be non-NULL");
    return AF_ERR_INVALID_ARG;
  }
  *out = nullptr;
  const af_ring_desc& d = *desc;
  if (d.n_slots <= 0 || d.max_pos <= 0 || d.n_layers < 0) {
    set_error("af_ring_create: n_slots and max_pos must be positive, n_layers >= 0");
    return AF_ERR_INVALID_ARG;
  }
  if (d.n_layers > 0) {
    if (d.dtype != AF_BF16 && d.dtype != AF_F32) {
      set_error("af_ring_create: dtype must be AF_BF16 or AF_F32");
      return AF_ERR_INVALID_ARG;
    }
    if (d.n_kv_heads <= 0 || (d.head_dim != 64 && d.head_dim != 128)) {
      set_error("af_ring_create: n_kv_heads > 0 and head_dim in {64, 128} required");
      return AF_ERR_UNSUPPORTED;
    }
  }
  af_ring* r = new (std::nothrow) af_ring();
  if (!r) {
    set_error("af_ring_create: host allocation failed");
    return AF_ERR_OOM;
  }
  r->d = d;
  r->owner.assign(d.n_slots, -1);
  r->len.assign(d.n_slots, 0);
  r->head = 0;
  if (d.n_layers > 0) {
    r->bytes = (size_t)d.n_layers * 2 * r->kv_region() * dtype_size(d.dtype);
    hipError_t e = hipMalloc(&r->kv, r->bytes);
    if (e != hipSuccess) {
      set_error("af_ring_create: hipMalloc(%zu) failed: %s", r->bytes, hipGetErrorString(e));
      delete r;
      return AF_ERR_OOM;
    }
    hipStream_t s = (hipStream_t)hip_stream;
    e = hipMemsetAsync(r->kv, 0, r->bytes, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) {
      set_error("af_ring_create: zero fill failed: %s", hipGetErrorString(e));
      (void)hipFree(r->kv);
      delete r;
      return AF_ERR_DEVICE;
    }
  }
  *out = r;
  return AF_OK;
}

extern "C" af_status af_ring_destroy(af_ring* ring) {
  clear_error();
  if (!ring) return AF_OK;
  if (ring->kv) {
    hipError_t e = hipFree(ring->kv);
    if (e != hipSuccess) {
      set_error("af_ring_destroy: hipFree failed: %s", hipGetErrorString(e));
      delete ring;
      return AF_ERR_DEVICE;
    }
  }
  delete ring;
  return AF_OK;
}

extern "C" af_status af_ring_reset(af_ring* ring) {
  clear_error();
  if (!ring) {
    set_error("af_ring_reset: NULL ring");
    return AF_ERR_INVALID_ARG;
  }
  ring->owner.assign(ring->d.n_slots, -1);
  ring->len.assign(ring->d.n_slots, 0);
  ring->head = 0;
  ring->slot_of.clear();
  return AF_OK;
}

extern "C" af_status af_ring_append(af_ring* ring, int64_t request_id, int32_t n_new, af_segment* out) {
  clear_error();
  if (!ring || !out) {
    set_error("af_ring_append: ring and out must be non-NULL");
    return AF_ERR_INVALID_ARG;
  }
  if (n_new <= 0 || request_id < 0) {
    set_error("af_ring_append: n_new must be positive and request_id >= 0 (got %d, %lld)", n_new,
              (long long)request_id);
    return AF_ERR_INVALID_ARG;
  }
  int32_t slot, pos0;
  auto it = ring->slot_of.find(request_id);
  if (it != ring->slot_of.end()) {  // continuation of a resident request
    slot = it->second;
    pos0 = ring->len[slot];
    if ((int64_t)pos0 + n_new > ring->d.max_pos) {
      set_error("af_ring_append: request %lld at position %d + %d exceeds max_pos %d", (long long)request_id, pos0,
                n_new, ring->d.max_pos);
      return AF_ERR_OUT_OF_RANGE;
    }
    ring->len[slot] = pos0 + n_new;
  } else {  // new request: next slot in rotation order
    slot = ring->head;
    if (ring->owner[slot] != -1) {
      set_error("af_ring_append: slot %d still owned by request %lld", slot, (long long)ring->owner[slot]);
      return AF_ERR_SLOT_BUSY;
    }
    if (n_new > ring->d.max_pos) {
      set_error("af_ring_append: %d positions exceed max_pos %d", n_new, ring->d.max_pos);
      return AF_ERR_OUT_OF_RANGE;
    }
    pos0 = 0;
    ring->owner[slot] = request_id;
    ring->len[slot] = n_new;
    ring->slot_of[request_id] = slot;
    ring->head = (slot + 1) % ring->d.n_slots;
  }
  out->q_start = 0;
  out->q_len = n_new;
  out->slot = slot;
  out->pos0 = pos0;
  out->request_id = request_id;
  out->flags = AF_SEG_EMIT;
  out->reserved = 0;
  return AF_OK;
}

extern "C" af_status af_ring_release(af_ring* ring, int64_t request_id) {
  clear_error();
  if (!ring) {
    set_error("af_ring_release: NULL ring");
    return AF_ERR_INVALID_ARG;
  }
  auto it = ring->slot_of.find(request_id);
  if (it == ring->slot_of.end()) {
    set_error("af_ring_release: request %lld owns no slot", (long long)request_id);
    return AF_ERR_UNKNOWN_REQUEST;
  }
  int32_t slot = it->second;
  ring->slot_of.erase(it);
  ring->owner[slot] = -1;
  ring->len[slot] = 0;
  return AF_OK;
}

extern "C" af_status af_ring_shift_stages(af_ring* ring, int32_t n_stages, void* hip_stream) {
  clear_error();
  if (!ring) {
    set_error("af_ring_shift_stages: NULL ring");
    return AF_ERR_INVALID_ARG;
  }
  if (n_stages < 2 || n_stages > ring->d.n_slots) {
    set_error("af_ring_shift_stages: n_stages %d outside [2, %d]", n_stages, ring->d.n_slots);
    return AF_ERR_INVALID_ARG;
  }
  if (ring->owner[n_stages - 1] != -1) {
    set_error("af_ring_shift_stages: slot %d (the last stage) still holds request %lld", n_stages - 1,
              (long long)ring->owner[n_stages - 1]);
    return AF_ERR_SLOT_BUSY;
  }
  const hipStream_t s = (hipStream_t)hip_stream;
  const size_t es = dtype_size(ring->d.dtype);
  const int H = ring->d.n_kv_heads, hd = ring->d.head_dim;
  for (int st = n_stages - 2; st >= 0; --st) {
    const int64_t rid = ring->owner[st];
    if (rid == -1) continue;
    const int n = ring->len[st];
    if (ring->kv && n > 0) {
      // runs: (layer, k|v) groups of H heads, each head's positions 0 .. n - 1 contiguous
      const size_t src = ring->offset(0, 0, st, 0, 0) * es, dst = ring->offset(0, 0, st + 1, 0, 0) * es;
      const size_t group = ring->kv_region() * es, head = (size_t)ring->d.max_pos * hd * es;
      hipError_t e = launch_run_copy(ring->kv, src, dst, 2 * ring->d.n_layers * H, H, group, head,
                                     (size_t)n * hd * es, s);
      if (e != hipSuccess) {
        set_error("af_ring_shift_stages: copy of slot %d failed: %s", st, hipGetErrorString(e));
        return AF_ERR_DEVICE;
      }
    }
    ring->owner[st + 1] = rid;
    ring->len[st + 1] = n;
    ring->slot_of[rid] = st + 1;
    ring->owner[st] = -1;
    ring->len[st] = 0;
  }
  ring->head = 0;
  return AF_OK;
}

extern "C" af_status af_ring_state(const af_ring* ring, int64_t* owners, int32_t* lens, int32_t* head) {
  clear_error();
  if (!ring) {
    set_error("af_ring_state: NULL ring");
    return AF_ERR_INVALID_ARG;
  }
  if (owners) std::memcpy(owners, ring->owner.data(), sizeof(int64_t) * ring->d.n_slots);
  if (lens) std::memcpy(lens, ring->len.data(), sizeof(int32_t) * ring->d.n_slots);
  if (head) *head = ring->head;
  return AF_OK;
}

static af_status ring_region_check(const af_ring* ring, int32_t layer, int32_t slot, int32_t pos0, int32_t n,
                                   const void* k, const void* v, const char* who) {
  if (!ring || !k || !v) {
    set_error("%s: ring, k and v must be non-NULL", who);
    return AF_ERR_INVALID_ARG;
  }
  if (!ring->kv) {
    set_error("%s: bookkeeping-only ring has no device storage", who);
    return AF_ERR_INVALID_ARG;
  }
  if (layer < 0 || layer >= ring->d.n_layers || slot < 0 || slot >= ring->d.n_slots || pos0 < 0 || n <= 0 ||
      (int64_t)pos0 + n > ring->d.max_pos) {
    set_error("%s: region (layer %d, slot %d, positions [%d, %d)) outside the ring", who, layer, slot, pos0, pos0 + n);
    return AF_ERR_OUT_OF_RANGE;
  }
  return AF_OK;
}

static af_status ring_copy(af_ring* ring, int32_t layer, int32_t slot, int32_t pos0, int32_t n, void* k, void* v,
                           bool to_ring, hipStream_t s) {
  const size_t es = dtype_size(ring->d.dtype);
  const int H = ring->d.n_kv_heads, hd = ring->d.head_dim;
  char* base = (char*)ring->kv;
  for (int kv_ = 0; kv_ < 2; ++kv_) {
    char* buf = (char*)(kv_ == 0 ? k : v);
    for (int h = 0; h < H; ++h) {
      char* ring_p = base + ring->offset(layer, kv_, slot, h, pos0) * es;
      char* buf_p = buf + (size_t)h * hd * es;
      // ring rows are contiguous positions of one head; caller rows interleave heads
      if (to_ring)
        AF_HIP(hipMemcpy2DAsync(ring_p, hd * es, buf_p, (size_t)H * hd * es, hd * es, n, hipMemcpyDeviceToDevice, s));
      else
        AF_HIP(hipMemcpy2DAsync(buf_p, (size_t)H * hd * es, ring_p, hd * es, hd * es, n, hipMemcpyDeviceToDevice, s));
    }
  }
  return AF_OK;
}

extern "C" af_status af_ring_write_kv(af_ring* ring, int32_t layer, int32_t slot, int32_t pos0, int32_t n,
                                      const void* k, const void* v, void* hip_stream) {
  clear_error();
  AF_TRY(ring_region_check(ring, layer, slot, pos0, n, k, v, "af_ring_write_kv"));
  return ring_copy(ring, layer, slot, pos0, n, (void*)k, (void*)v, true, (hipStream_t)hip_stream);
}

extern "C" af_status af_ring_read_kv(af_ring* ring, int32_t layer, int32_t slot, int32_t pos0, int32_t n, void* k,
                                     void* v, void* hip_stream) {
  clear_error();
  AF_TRY(ring_region_check(ring, layer, slot, pos0, n, k, v, "af_ring_read_kv"));
  return ring_copy(ring, layer, slot, pos0, n, k, v, false, (hipStream_t)hip_stream);
}

extern "C" af_status af_ring_copy_kv(const af_ring* src, int32_t src_layer, int32_t src_slot, af_ring* dst,
                                     int32_t dst_layer, int32_t dst_slot, int32_t pos0, int32_t n, void* hip_stream) {
  clear_error();
  const int dummy = 0;
  AF_TRY(ring_region_check(src, src_layer, src_slot, pos0, n, &dummy, &dummy, "af_ring_copy_kv (source)"));
  AF_TRY(ring_region_check(dst, dst_layer, dst_slot, pos0, n, &dummy, &dummy, "af_ring_copy_kv (destination)"));
  if (src->d.n_kv_heads != dst->d.n_kv_heads || src->d.head_dim != dst->d.head_dim || src->d.dtype != dst->d.dtype) {
    set_error("af_ring_copy_kv: rings differ in heads, head_dim or dtype");
    return AF_ERR_INVALID_ARG;
  }
  if (src == dst && src_layer == dst_layer && src_slot == dst_slot) return AF_OK;  // the region onto itself
  const size_t es = dtype_size(src->d.dtype);
  const int H = src->d.n_kv_heads, hd = src->d.head_dim;
  // runs (kv, head): positions [pos0, pos0 + n) of one head are contiguous in a ring
  const CopyStrides st{(src->offset(0, 1, 0, 0, 0) - src->offset(0, 0, 0, 0, 0)) * es, (size_t)src->d.max_pos * hd * es,
                       (dst->offset(0, 1, 0, 0, 0) - dst->offset(0, 0, 0, 0, 0)) * es, (size_t)dst->d.max_pos * hd * es};
  const char* from = (const char*)src->kv + src->offset(src_layer, 0, src_slot, 0, pos0) * es;
  char* to = (char*)dst->kv + dst->offset(dst_layer, 0, dst_slot, 0, pos0) * es;
  AF_HIP(launch_copy_runs(from, to, 2 * H, H, st, (size_t)n * hd * es, (hipStream_t)hip_stream));
  return AF_OK;
}
