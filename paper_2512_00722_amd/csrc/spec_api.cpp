// C ABI of the decode-step hot path: argument validation (host only, before
// any HIP call), workspace carve-up and kernel dispatch on the caller's
// stream.  The library holds no state except a per-thread last HIP error.
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

#include "../../include/spec.h"
#include "internal.h"

namespace spec {
size_t elastic_plan_lds_bytes(const Dims& d);
}

namespace {

thread_local int g_last_hip_error = 0;

constexpr int kMaxElasticLcap = 245760;  // two LDS bitmaps of L_cap bits <= 60 KiB

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
bool aligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) == 0; }

// Query heads per KV head: a power of two up to 128 (more than 16 run as
// several 16-head column groups over the same KV head).
bool is_pow2_group(int g) { return g >= 1 && g <= 128 && (g & (g - 1)) == 0; }

spec_status resolve(const spec_dims* dm, spec::Dims* o) {
  if (!dm) return SPEC_ERR_INVALID;
  if (dm->B <= 0 || dm->L_cap <= 0 || dm->L_max <= 0 || dm->k_max <= 0 || dm->H_r <= 0 ||
      dm->d_r <= 0 || dm->n_layers <= 0 || dm->H_q <= 0 || dm->H_kv <= 0 || dm->d <= 0)
    return SPEC_ERR_INVALID;
  if (dm->reserved != 0) return SPEC_ERR_INVALID;
  if (dm->L_max > dm->L_cap || dm->k_max > dm->L_max) return SPEC_ERR_INVALID;
  if (dm->H_q % dm->H_kv != 0) return SPEC_ERR_INVALID;
  if (dm->kr_stride_b < 0 || dm->kv_stride_layer < 0 || dm->kv_stride_b < 0)
    return SPEC_ERR_INVALID;
  if (!(isfinite(dm->scale_r) && isfinite(dm->scale)) || dm->scale_r < 0.f || dm->scale < 0.f)
    return SPEC_ERR_INVALID;
  // One token set per sequence (the heads' weights summed), or one per KV
  // head (the maximum over the retrieval heads of its group).
  if (dm->n_sets != 1 && dm->n_sets != dm->H_kv) return SPEC_ERR_UNSUPPORTED;
  if (dm->n_sets > 1 && (dm->H_r % dm->n_sets != 0 || (int64_t)dm->B * dm->n_sets > 65535))
    return SPEC_ERR_UNSUPPORTED;
  if (dm->d != 128) return SPEC_ERR_UNSUPPORTED;
  if (dm->d_r != 64 && dm->d_r != 128) return SPEC_ERR_UNSUPPORTED;
  if (dm->H_r > 16) return SPEC_ERR_UNSUPPORTED;
  if (dm->H_kv > 16) return SPEC_ERR_UNSUPPORTED;
  if (!is_pow2_group(dm->H_q / dm->H_kv)) return SPEC_ERR_UNSUPPORTED;
  if (dm->B > 65535 || dm->n_layers > 65535) return SPEC_ERR_UNSUPPORTED;

  const int64_t kr_row = (int64_t)dm->L_cap * dm->H_r * dm->d_r;
  const int64_t kv_row = (int64_t)dm->L_cap * dm->H_kv * dm->d;
  o->B = dm->B;
  o->L_cap = dm->L_cap;
  o->L_max = dm->L_max;
  o->k_max = dm->k_max;
  o->H_r = dm->H_r;
  o->d_r = dm->d_r;
  o->n_layers = dm->n_layers;
  o->H_q = dm->H_q;
  o->H_kv = dm->H_kv;
  o->d = dm->d;
  o->G = dm->H_q / dm->H_kv;
  o->n_sets = dm->n_sets;
  o->kr_stride_b = dm->kr_stride_b ? dm->kr_stride_b : kr_row;
  o->kv_stride_b = dm->kv_stride_b ? dm->kv_stride_b : kv_row;
  o->kv_stride_layer = dm->kv_stride_layer ? dm->kv_stride_layer : (int64_t)dm->B * o->kv_stride_b;
  if (o->kr_stride_b < kr_row || o->kr_stride_b % 8) return SPEC_ERR_INVALID;
  if (o->kv_stride_b < kv_row || o->kv_stride_b % 8) return SPEC_ERR_INVALID;
  if (o->kv_stride_layer < kv_row || o->kv_stride_layer % 8) return SPEC_ERR_INVALID;
  o->scale_r = dm->scale_r > 0.f ? dm->scale_r : 1.0f / sqrtf((float)dm->d_r);
  o->scale = dm->scale > 0.f ? dm->scale : 1.0f / sqrtf((float)dm->d);
  return SPEC_OK;
}

// Attention workspace large enough for a launch over any number of layers
// up to d.n_layers (the offloaded step attends its device layers in one
// launch and each offloaded layer in one of its own).
size_t attn_ws_any_layers(const spec::Dims& d) {
  size_t m = 0;
  spec::Dims e = d;
  for (int n = 1; n <= d.n_layers; ++n) {
    e.n_layers = n;
    const size_t b = spec::attn_ws_bytes(e);
    if (b > m) m = b;
  }
  return m;
}

size_t ws_bytes_for(const spec::Dims& d, spec_op op) {
  switch (op) {
    case SPEC_OP_SCORE: return spec::score_ws_bytes(d);
    case SPEC_OP_TOPK: return spec::topk_ws_bytes(d);
    case SPEC_OP_GATHER: return 0;
    case SPEC_OP_ATTN: return spec::attn_ws_bytes(d);
    case SPEC_OP_DELTA: return spec::delta_ws_bytes(d);
    case SPEC_OP_FRONTEND: return spec::front_ws_bytes(d);
    case SPEC_OP_STEP:
      return spec::align_up(sizeof(float) * (size_t)d.B * d.n_sets * d.L_max) +
             spec::score_ws_bytes(d) +
             spec::topk_ws_bytes(d) + spec::attn_ws_bytes(d) + spec::delta_ws_bytes(d);
    case SPEC_OP_OFFLOAD:
      return spec::align_up(sizeof(float) * (size_t)d.B * d.n_sets * d.L_max) +
             spec::score_ws_bytes(d) + spec::topk_ws_bytes(d) + attn_ws_any_layers(d) +
             spec::delta_ws_bytes(d);
  }
  return 0;
}

spec_status check_ws(const spec::Dims& d, spec_op op, const void* ws, size_t ws_bytes) {
  const size_t need = ws_bytes_for(d, op);
  if (need == 0) return SPEC_OK;
  if (!ws || ws_bytes < need) return SPEC_ERR_WORKSPACE;
  if (!aligned16(ws)) return SPEC_ERR_INVALID;
  return SPEC_OK;
}

spec_status hip_status(hipError_t e) {
  if (e == hipSuccess) return SPEC_OK;
  g_last_hip_error = (int)e;
  return SPEC_ERR_HIP;
}

hipStream_t as_stream(spec_stream s) { return reinterpret_cast<hipStream_t>(s); }

// ---- SPEC_DEBUG=1 ---------------------------------------------------------
// Read at every call.  Before a launch, the device-resident lengths and
// indices are copied to the host (a synchronising copy on the caller's
// stream) and values the kernels would clamp are reported as
// SPEC_ERR_INVALID, with nothing enqueued; after the launch the stream is
// synchronised and an asynchronous failure is reported as SPEC_ERR_HIP.
// For debugging: the calls then synchronise and cannot be graph-captured.
bool debug_on() {
  const char* e = getenv("SPEC_DEBUG");
  return e && e[0] == '1' && e[1] == 0;
}

template <class T>
bool d2h(std::vector<T>& h, const T* p, size_t n, hipStream_t s) {
  h.resize(n);
  if (n == 0) return true;
  if (hipMemcpyAsync(h.data(), p, n * sizeof(T), hipMemcpyDeviceToHost, s) != hipSuccess)
    return false;
  return hipStreamSynchronize(s) == hipSuccess;
}

// seq_lens[b] in [0, L_max]; ks[b] >= 0 (either pointer may be null).
spec_status debug_lengths(const spec::Dims& d, const int32_t* seq_lens, const int32_t* ks,
                          hipStream_t s) {
  std::vector<int32_t> h;
  if (seq_lens) {
    if (!d2h(h, seq_lens, d.B, s)) return SPEC_ERR_HIP;
    for (int32_t v : h)
      if (v < 0 || v > d.L_max) return SPEC_ERR_INVALID;
  }
  if (ks) {
    if (!d2h(h, ks, d.B, s)) return SPEC_ERR_HIP;
    for (int32_t v : h)
      if (v < 0) return SPEC_ERR_INVALID;
  }
  return SPEC_OK;
}

// counts[b] in [0, k_max]; with idx, idx[b][set][j] in [0, limit) for j < counts[b].
spec_status debug_selection(int B, int k_max, int n_sets, const int32_t* idx,
                            const int32_t* counts, int limit, hipStream_t s) {
  std::vector<int32_t> c, ix;
  if (!d2h(c, counts, (size_t)B, s)) return SPEC_ERR_HIP;
  for (int32_t v : c)
    if (v < 0 || v > k_max) return SPEC_ERR_INVALID;
  if (!idx) return SPEC_OK;
  if (!d2h(ix, idx, (size_t)B * n_sets * k_max, s)) return SPEC_ERR_HIP;
  for (int b = 0; b < B; ++b)
    for (int g = 0; g < n_sets; ++g)
      for (int j = 0; j < c[b]; ++j) {
        const int32_t v = ix[((size_t)b * n_sets + g) * k_max + j];
        if (v < 0 || v >= limit) return SPEC_ERR_INVALID;
      }
  return SPEC_OK;
}

// Elastic slot sources: -1 (read the slot) or a token index of the caches.
spec_status debug_slot_src(const spec::Dims& d, const int32_t* slot_src, hipStream_t s) {
  std::vector<int32_t> h;
  if (!d2h(h, slot_src, (size_t)d.B * d.k_max, s)) return SPEC_ERR_HIP;
  for (int32_t v : h)
    if (v < -1 || v >= d.L_cap) return SPEC_ERR_INVALID;
  return SPEC_OK;
}

// How the fused step applies an elastic update.  By default the attention
// loads the rows of mostly-new sequences itself and the others are copied
// first; SPEC_ELASTIC_PATH=copy copies every update before a compact
// attention (spec_delta_gather's path), SPEC_ELASTIC_PATH=fused lets the
// attention load every update (tests compare the three).
enum { kElasticAuto = 0, kElasticCopy = 1, kElasticFused = 2 };
int elastic_path() {
  const char* e = getenv("SPEC_ELASTIC_PATH");
  if (e && strcmp(e, "copy") == 0) return kElasticCopy;
  if (e && strcmp(e, "fused") == 0) return kElasticFused;
  return kElasticAuto;
}

// After a launch: in debug mode wait for the stream and report its status.
spec_status finish(spec_status st, hipStream_t s) {
  if (st != SPEC_OK || !debug_on()) return st;
  hipError_t e = hipStreamSynchronize(s);
  if (e == hipSuccess) e = hipGetLastError();
  return hip_status(e);
}

spec_status check_elastic(const spec::Dims& d, const spec_elastic* el) {
  if (!el || !el->slot_tok || !el->kbuf || !el->vbuf || !el->n_changed || !el->slot_src)
    return SPEC_ERR_INVALID;
  // the compact slot buffers hold one token per slot for every KV head
  if (d.n_sets != 1) return SPEC_ERR_UNSUPPORTED;
  if (!aligned4(el->slot_tok) || !aligned4(el->n_changed) || !aligned4(el->slot_src) ||
      !aligned16(el->kbuf) || !aligned16(el->vbuf))
    return SPEC_ERR_INVALID;
  if (d.L_cap > kMaxElasticLcap) return SPEC_ERR_UNSUPPORTED;
  return SPEC_OK;
}

// Offloaded KV in pinned host memory: both pointers must be host memory the
// GPU can read (hipHostMalloc); the kernels use their device addresses.
// Strides default as for the device cache and are checked the same way.
struct HostKv {
  const uint16_t* k;
  const uint16_t* v;
  int64_t stride_layer, stride_b;
};

spec_status resolve_host_kv(const spec::Dims& d, const spec_host_kv* h, HostKv* o) {
  if (!h || !h->k || !h->v) return SPEC_ERR_INVALID;
  if (!aligned16(h->k) || !aligned16(h->v)) return SPEC_ERR_INVALID;
  if (h->stride_layer < 0 || h->stride_b < 0) return SPEC_ERR_INVALID;
  const int64_t row = (int64_t)d.L_cap * d.H_kv * d.d;
  o->stride_b = h->stride_b ? h->stride_b : row;
  o->stride_layer = h->stride_layer ? h->stride_layer : (int64_t)d.B * o->stride_b;
  if (o->stride_b < row || o->stride_b % 8 || o->stride_layer < row || o->stride_layer % 8)
    return SPEC_ERR_INVALID;
  const void* src[2] = {h->k, h->v};
  const uint16_t* dev[2] = {nullptr, nullptr};
  for (int i = 0; i < 2; ++i) {
    hipPointerAttribute_t at;
    if (hipPointerGetAttributes(&at, src[i]) != hipSuccess) {
      (void)hipGetLastError();  // an unknown (pageable) pointer: clear the error it leaves
      return SPEC_ERR_INVALID;
    }
    if (at.type != hipMemoryTypeHost || !at.devicePointer) return SPEC_ERR_INVALID;
    dev[i] = static_cast<const uint16_t*>(at.devicePointer);
  }
  o->k = dev[0];
  o->v = dev[1];
  return SPEC_OK;
}

// The host-to-device loads of n_off offloaded layers after the slot plan
// (already enqueued on s): with a copy stream, forked at ready[n_off] and
// each layer's rows followed by ready[l] on it; else on s.
spec_status enqueue_host_loads(const spec::Dims& d_off, const HostKv& hk, const spec_elastic* el,
                               const void* ws_delta, int n_off, hipStream_t s, hipStream_t cs,
                               void* const* ready) {
  const hipStream_t q = cs ? cs : s;
  hipError_t e;
  if (cs) {
    hipEvent_t fork = static_cast<hipEvent_t>(ready[n_off]);
    if ((e = hipEventRecord(fork, s)) != hipSuccess) return hip_status(e);
    if ((e = hipStreamWaitEvent(cs, fork, 0)) != hipSuccess) return hip_status(e);
  }
  const int64_t slot_layer = (int64_t)d_off.B * d_off.k_max * d_off.H_kv * d_off.d;
  for (int l = 0; l < n_off; ++l) {
    e = spec::launch_delta_copy(d_off, hk.k + (int64_t)l * hk.stride_layer,
                                hk.v + (int64_t)l * hk.stride_layer, hk.stride_layer, hk.stride_b,
                                1, el->n_changed, el->kbuf + l * slot_layer,
                                el->vbuf + l * slot_layer, ws_delta, q, nullptr,
                                /*from_host=*/true);
    if (e != hipSuccess) return hip_status(e);
    if (ready && (e = hipEventRecord(static_cast<hipEvent_t>(ready[l]), q)) != hipSuccess)
      return hip_status(e);
  }
  return SPEC_OK;
}

spec_status resolve_frontend(const spec_frontend* fe, spec::FrontDims* f) {
  if (!fe || fe->reserved != 0) return SPEC_ERR_INVALID;
  if (fe->vocab <= 0 || fe->hidden <= 0) return SPEC_ERR_INVALID;
  if (!isfinite(fe->rope_base) || !(fe->rope_base > 0.f) || !isfinite(fe->yarn_scale))
    return SPEC_ERR_INVALID;
  if (fe->hidden % 128 != 0) return SPEC_ERR_UNSUPPORTED;
  f->vocab = fe->vocab;
  f->hidden = fe->hidden;
  f->base = fe->rope_base;
  f->scale = fe->yarn_scale;
  f->orig_ctx = fe->yarn_orig_ctx;
  f->alpha = fe->yarn_alpha;
  f->beta = fe->yarn_beta;
  if (fe->yarn_scale > 1.f) {
    if (fe->yarn_orig_ctx <= 0) return SPEC_ERR_INVALID;
    if (fe->yarn_alpha == 0.f && fe->yarn_beta == 0.f) {
      f->alpha = 1.f;
      f->beta = 32.f;
    }
    if (!isfinite(f->alpha) || !isfinite(f->beta) || !(f->alpha < f->beta))
      return SPEC_ERR_INVALID;
  }
  return SPEC_OK;
}

spec_status resolve_mla(const spec_mla_dims* dm, spec::MlaDims* o) {
  if (!dm || dm->reserved != 0 || dm->reserved2 != 0) return SPEC_ERR_INVALID;
  if (dm->B <= 0 || dm->L_cap <= 0 || dm->k_max <= 0 || dm->n_layers <= 0 || dm->H <= 0 ||
      dm->d_c <= 0 || dm->d_rope <= 0 || dm->d_nope <= 0 || dm->d_v <= 0)
    return SPEC_ERR_INVALID;
  if (dm->k_max > dm->L_cap) return SPEC_ERR_INVALID;
  if (dm->ckv_stride_layer < 0 || dm->ckv_stride_b < 0) return SPEC_ERR_INVALID;
  if (!isfinite(dm->scale) || dm->scale < 0.f) return SPEC_ERR_INVALID;
  if (dm->d_c != 512 || dm->d_rope != 64 || dm->d_nope != 128 || dm->d_v != 128)
    return SPEC_ERR_UNSUPPORTED;
  if (dm->H != 64 && dm->H != 128) return SPEC_ERR_UNSUPPORTED;
  if (dm->k_max > 32768 || dm->B > 65535) return SPEC_ERR_UNSUPPORTED;
  if ((int64_t)dm->n_layers * dm->H > INT32_MAX || (int64_t)dm->n_layers * dm->B > 1 << 24)
    return SPEC_ERR_UNSUPPORTED;
  const int64_t row = (int64_t)dm->L_cap * (dm->d_c + dm->d_rope);
  o->B = dm->B;
  o->L_cap = dm->L_cap;
  o->k_max = dm->k_max;
  o->n_layers = dm->n_layers;
  o->H = dm->H;
  o->stride_b = dm->ckv_stride_b ? dm->ckv_stride_b : row;
  o->stride_layer = dm->ckv_stride_layer ? dm->ckv_stride_layer : (int64_t)dm->B * o->stride_b;
  if (o->stride_b < row || o->stride_b % 8) return SPEC_ERR_INVALID;
  if (o->stride_layer < row || o->stride_layer % 8) return SPEC_ERR_INVALID;
  o->scale = dm->scale > 0.f ? dm->scale : 1.0f / sqrtf((float)(dm->d_nope + dm->d_rope));
  return SPEC_OK;
}


// Host checks shared by the two step entry points (before any HIP call).
spec_status check_step(const spec_dims* dm, spec::Dims* d, const uint16_t* q_r,
                       const uint16_t* k_r, const int32_t* seq_lens, const int32_t* ks,
                       const uint16_t* q, const uint16_t* k_cache, const uint16_t* v_cache,
                       const int32_t* idx_out, const int32_t* counts_out, const float* out,
                       const float* lse, const float* scores_out, const spec_elastic* el) {
  spec_status st = resolve(dm, d);
  if (st != SPEC_OK) return st;
  if (!q_r || !k_r || !seq_lens || !ks || !q || !k_cache || !v_cache || !idx_out ||
      !counts_out || !out)
    return SPEC_ERR_INVALID;
  if (!aligned16(q_r) || !aligned16(k_r) || !aligned4(seq_lens) || !aligned4(ks) ||
      !aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned4(idx_out) ||
      !aligned4(counts_out) || !aligned16(out) || (lse && !aligned4(lse)) ||
      (scores_out && !aligned4(scores_out)))
    return SPEC_ERR_INVALID;
  if (el && (st = check_elastic(*d, el)) != SPEC_OK) return st;
  return SPEC_OK;
}

// The step's launches on workspace `ws` (spec_workspace_size(SPEC_OP_STEP)
// bytes, carved as below).  Every region is written before it is read
// within the call (the histogram is cleared by the first kernel), so the
// workspace need not start zeroed.
spec_status run_step(const spec::Dims& d, const uint16_t* q_r, const uint16_t* k_r,
                     const int32_t* seq_lens, const int32_t* ks, const uint16_t* q,
                     const uint16_t* k_cache, const uint16_t* v_cache, int32_t* idx_out,
                     int32_t* counts_out, float* out, float* lse, float* scores_out,
                     const spec_elastic* el, void* ws, hipStream_t s) {
  char* p = static_cast<char*>(ws);
  float* scores = reinterpret_cast<float*>(p);
  p += spec::align_up(sizeof(float) * (size_t)d.B * d.n_sets * d.L_max);
  void* ws_score = p;
  p += spec::score_ws_bytes(d);
  void* ws_topk = p;
  p += spec::topk_ws_bytes(d);
  void* ws_attn = p;
  p += spec::attn_ws_bytes(d);
  void* ws_delta = p;

  hipError_t e = spec::launch_score_select(d, q_r, k_r, seq_lens, ks, scores_out, scores,
                                           idx_out, counts_out, ws_score, ws_topk, s);
  if (e != hipSuccess) return hip_status(e);
  const int path = el ? elastic_path() : 0;
  if (el && path == kElasticCopy) {  // the update's copy, then compact attention
    e = spec::launch_delta(d, idx_out, counts_out, k_cache, v_cache, el->slot_tok, el->slot_src,
                           el->kbuf, el->vbuf, el->n_changed, ws_delta, s);
    if (e != hipSuccess) return hip_status(e);
    e = spec::launch_attn(d, q, el->kbuf, el->vbuf, nullptr, counts_out, out, lse, ws_attn, s);
  } else if (el) {
    // The plan marks the sequences whose update is mostly new (a full
    // reload): the attention loads their rows from the caches into the
    // slots as it streams them.  The other sequences' rows are copied first
    // and the attention only reads the slots.
    const int pct = path == kElasticFused ? 0 : spec::kElasticFusePct;
    e = spec::launch_delta_plan(d, idx_out, counts_out, el->slot_tok, el->slot_src,
                                el->n_changed, ws_delta, s, pct);
    if (e != hipSuccess) return hip_status(e);
    const int32_t* fused = spec::delta_ws_fused(d, ws_delta);
    e = spec::launch_delta_copy(d, k_cache, v_cache, d.kv_stride_layer, d.kv_stride_b,
                                d.n_layers, el->n_changed, el->kbuf, el->vbuf, ws_delta, s,
                                fused);
    if (e != hipSuccess) return hip_status(e);
    e = spec::launch_attn_elastic(d, q, k_cache, v_cache, el->kbuf, el->vbuf, el->slot_src,
                                  counts_out, out, lse, ws_attn, s, fused);
  } else {
    e = spec::launch_attn(d, q, k_cache, v_cache, idx_out, counts_out, out, lse, ws_attn, s);
  }
  return finish(hip_status(e), s);
}

}  // namespace

extern "C" {

spec_status spec_mla_workspace_size(const spec_mla_dims* dm, size_t* bytes) {
  if (!bytes) return SPEC_ERR_INVALID;
  spec::MlaDims d;
  const spec_status st = resolve_mla(dm, &d);
  if (st != SPEC_OK) return st;
  *bytes = spec::mla_ws_bytes(d);
  return SPEC_OK;
}

spec_status spec_mla_sparse_decode_attn(const spec_mla_dims* dm, const uint16_t* q,
                                        const uint16_t* ckv, const uint16_t* w_uk,
                                        const uint16_t* w_uv, const int32_t* idx,
                                        const int32_t* counts, float* out, float* lse, void* ws,
                                        size_t ws_bytes, spec_stream stream) {
  spec::MlaDims d;
  spec_status st = resolve_mla(dm, &d);
  if (st != SPEC_OK) return st;
  if (!q || !ckv || !w_uk || !w_uv || !idx || !counts || !out) return SPEC_ERR_INVALID;
  if (!aligned16(q) || !aligned16(ckv) || !aligned16(w_uk) || !aligned16(w_uv) ||
      !aligned4(idx) || !aligned4(counts) || !aligned16(out) || (lse && !aligned4(lse)))
    return SPEC_ERR_INVALID;
  const size_t need = spec::mla_ws_bytes(d);
  if (!ws || ws_bytes < need) return SPEC_ERR_WORKSPACE;
  if (!aligned16(ws)) return SPEC_ERR_INVALID;
  if (debug_on() && (st = debug_selection(d.B, d.k_max, 1, idx, counts, d.L_cap,
                                          as_stream(stream))) != SPEC_OK)
    return st;
  return finish(hip_status(spec::launch_mla(d, q, ckv, w_uk, w_uv, idx, counts, out, lse, ws,
                                            as_stream(stream))),
                as_stream(stream));
}

spec_status spec_workspace_size(const spec_dims* dm, spec_op op, size_t* bytes) {
  if (!bytes) return SPEC_ERR_INVALID;
  if ((int)op < SPEC_OP_SCORE || (int)op > SPEC_OP_OFFLOAD) return SPEC_ERR_INVALID;
  spec::Dims d;
  const spec_status st = resolve(dm, &d);
  if (st != SPEC_OK) return st;
  *bytes = ws_bytes_for(d, op);
  return SPEC_OK;
}

spec_status spec_score(const spec_dims* dm, const uint16_t* q_r, const uint16_t* k_r,
                       const int32_t* seq_lens, float* scores, void* ws, size_t ws_bytes,
                       spec_stream stream) {
  spec::Dims d;
  spec_status st = resolve(dm, &d);
  if (st != SPEC_OK) return st;
  if (!q_r || !k_r || !seq_lens || !scores) return SPEC_ERR_INVALID;
  if (!aligned16(q_r) || !aligned16(k_r) || !aligned4(seq_lens) || !aligned4(scores))
    return SPEC_ERR_INVALID;
  if ((st = check_ws(d, SPEC_OP_SCORE, ws, ws_bytes)) != SPEC_OK) return st;
  if (debug_on() && (st = debug_lengths(d, seq_lens, nullptr, as_stream(stream))) != SPEC_OK)
    return st;
  return finish(
      hip_status(spec::launch_score(d, q_r, k_r, seq_lens, scores, ws, as_stream(stream))),
      as_stream(stream));
}

spec_status spec_topk(const spec_dims* dm, const float* scores, const int32_t* seq_lens,
                      const int32_t* ks, int32_t* idx, int32_t* counts, void* ws,
                      size_t ws_bytes, spec_stream stream) {
  spec::Dims d;
  spec_status st = resolve(dm, &d);
  if (st != SPEC_OK) return st;
  if (!scores || !seq_lens || !ks || !idx) return SPEC_ERR_INVALID;
  if (!aligned4(scores) || !aligned4(seq_lens) || !aligned4(ks) || !aligned4(idx) ||
      (counts && !aligned4(counts)))
    return SPEC_ERR_INVALID;
  if ((st = check_ws(d, SPEC_OP_TOPK, ws, ws_bytes)) != SPEC_OK) return st;
  if (debug_on() && (st = debug_lengths(d, seq_lens, ks, as_stream(stream))) != SPEC_OK) return st;
  return finish(hip_status(spec::launch_topk(d, scores, seq_lens, ks, idx, counts, ws,
                                             as_stream(stream))),
                as_stream(stream));
}

spec_status spec_gather(const spec_dims* dm, const uint16_t* k_cache, const uint16_t* v_cache,
                        const int32_t* idx, const int32_t* counts, uint16_t* k_sel,
                        uint16_t* v_sel, spec_stream stream) {
  spec::Dims d;
  spec_status st = resolve(dm, &d);
  if (st != SPEC_OK) return st;
  if (!k_cache || !v_cache || !idx || !counts || !k_sel || !v_sel) return SPEC_ERR_INVALID;
  if (!aligned16(k_cache) || !aligned16(v_cache) || !aligned16(k_sel) || !aligned16(v_sel) ||
      !aligned4(idx) || !aligned4(counts))
    return SPEC_ERR_INVALID;
  if (debug_on() && (st = debug_selection(d.B, d.k_max, d.n_sets, idx, counts, d.L_cap,
                                          as_stream(stream))) != SPEC_OK)
    return st;
  return finish(hip_status(spec::launch_gather(d, k_cache, v_cache, idx, counts, k_sel, v_sel,
                                               as_stream(stream))),
                as_stream(stream));
}

spec_status spec_sparse_decode_attn(const spec_dims* dm, const uint16_t* q, const uint16_t* k,
                                    const uint16_t* v, const int32_t* idx,
                                    const int32_t* counts, float* out, float* lse, void* ws,
                                    size_t ws_bytes, spec_stream stream) {
  spec::Dims d;
  spec_status st = resolve(dm, &d);
  if (st != SPEC_OK) return st;
  if (!q || !k || !v || !counts || !out) return SPEC_ERR_INVALID;
  if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned4(counts) ||
      !aligned16(out) || (idx && !aligned4(idx)) || (lse && !aligned4(lse)))
    return SPEC_ERR_INVALID;
  if ((st = check_ws(d, SPEC_OP_ATTN, ws, ws_bytes)) != SPEC_OK) return st;
  if (debug_on() && (st = debug_selection(d.B, d.k_max, d.n_sets, idx, counts, d.L_cap,
                                          as_stream(stream))) != SPEC_OK)
    return st;
  return finish(hip_status(spec::launch_attn(d, q, k, v, idx, counts, out, lse, ws,
                                             as_stream(stream))),
                as_stream(stream));
}

spec_status spec_delta_gather(const spec_dims* dm, const int32_t* idx_now,
                              const int32_t* counts, const uint16_t* k_cache,
                              const uint16_t* v_cache, const spec_elastic* el, void* ws,
                              size_t ws_bytes, spec_stream stream) {
  spec::Dims d;
  spec_status st = resolve(dm, &d);
  if (st != SPEC_OK) return st;
  if (!idx_now || !counts || !k_cache || !v_cache) return SPEC_ERR_INVALID;
  if (!aligned4(idx_now) || !aligned4(counts) || !aligned16(k_cache) || !aligned16(v_cache))
    return SPEC_ERR_INVALID;
  if ((st = check_elastic(d, el)) != SPEC_OK) return st;
  if ((st = check_ws(d, SPEC_OP_DELTA, ws, ws_bytes)) != SPEC_OK) return st;
  if (debug_on() && (st = debug_selection(d.B, d.k_max, 1, idx_now, counts, d.L_cap,
                                          as_stream(stream))) != SPEC_OK)
    return st;
  return finish(hip_status(spec::launch_delta(d, idx_now, counts, k_cache, v_cache,
                                              el->slot_tok, el->slot_src, el->kbuf, el->vbuf,
                                              el->n_changed, ws, as_stream(stream))),
                as_stream(stream));
}

spec_status spec_sparse_decode_attn_elastic(const spec_dims* dm, const uint16_t* q,
                                            const uint16_t* k_cache, const uint16_t* v_cache,
                                            const spec_elastic* el, const int32_t* counts,
                                            float* out, float* lse, void* ws, size_t ws_bytes,
                                            spec_stream stream) {
  spec::Dims d;
  spec_status st = resolve(dm, &d);
  if (st != SPEC_OK) return st;
  if (!q || !k_cache || !v_cache || !counts || !out) return SPEC_ERR_INVALID;
  if (!aligned16(q) || !aligned16(k_cache) || !aligned16(v_cache) || !aligned4(counts) ||
      !aligned16(out) || (lse && !aligned4(lse)))
    return SPEC_ERR_INVALID;
  if ((st = check_elastic(d, el)) != SPEC_OK) return st;
  if ((st = check_ws(d, SPEC_OP_ATTN, ws, ws_bytes)) != SPEC_OK) return st;
  if (debug_on() &&
      ((st = debug_selection(d.B, d.k_max, 1, nullptr, counts, d.L_cap, as_stream(stream))) !=
           SPEC_OK ||
       (st = debug_slot_src(d, el->slot_src, as_stream(stream))) != SPEC_OK))
    return st;
  return finish(hip_status(spec::launch_attn_elastic(d, q, k_cache, v_cache, el->kbuf, el->vbuf,
                                                     el->slot_src, counts, out, lse, ws,
                                                     as_stream(stream))),
                as_stream(stream));
}

spec_status spec_step(const spec_dims* dm, const uint16_t* q_r, const uint16_t* k_r,
                      const int32_t* seq_lens, const int32_t* ks, const uint16_t* q,
                      const uint16_t* k_cache, const uint16_t* v_cache, int32_t* idx_out,
                      int32_t* counts_out, float* out, float* lse, float* scores_out,
                      const spec_elastic* el, void* ws, size_t ws_bytes,
                      spec_stream stream) {
  spec::Dims d;
  spec_status st = check_step(dm, &d, q_r, k_r, seq_lens, ks, q, k_cache, v_cache, idx_out,
                              counts_out, out, lse, scores_out, el);
  if (st != SPEC_OK) return st;
  if ((st = check_ws(d, SPEC_OP_STEP, ws, ws_bytes)) != SPEC_OK) return st;
  if (debug_on() && (st = debug_lengths(d, seq_lens, ks, as_stream(stream))) != SPEC_OK) return st;
  return run_step(d, q_r, k_r, seq_lens, ks, q, k_cache, v_cache, idx_out, counts_out, out, lse,
                  scores_out, el, ws, as_stream(stream));
}

spec_status spec_step_noalloc(const spec_dims* dm, const uint16_t* q_r, const uint16_t* k_r,
                              const int32_t* seq_lens, const int32_t* ks, const uint16_t* q,
                              const uint16_t* k_cache, const uint16_t* v_cache,
                              int32_t* idx_out, int32_t* counts_out, float* out, float* lse,
                              float* scores_out, const spec_elastic* el, spec_stream stream) {
  spec::Dims d;
  spec_status st = check_step(dm, &d, q_r, k_r, seq_lens, ks, q, k_cache, v_cache, idx_out,
                              counts_out, out, lse, scores_out, el);
  if (st != SPEC_OK) return st;
  if (ws_bytes_for(d, SPEC_OP_STEP) > spec::kStaticScratchBytes) return SPEC_ERR_TOO_LARGE;
  if (debug_on() && (st = debug_lengths(d, seq_lens, ks, as_stream(stream))) != SPEC_OK) return st;
  void* ws = nullptr;  // the device address of this GPU's static scratch
  const hipError_t e = spec::static_scratch(&ws);
  if (e != hipSuccess) return hip_status(e);
  return run_step(d, q_r, k_r, seq_lens, ks, q, k_cache, v_cache, idx_out, counts_out, out, lse,
                  scores_out, el, ws, as_stream(stream));
}

size_t spec_step_noalloc_max_bytes(void) { return spec::kStaticScratchBytes; }

spec_status spec_offload_load(const spec_dims* dm, const int32_t* idx_now, const int32_t* counts,
                              const spec_host_kv* host, const spec_elastic* el, void* ws,
                              size_t ws_bytes, spec_stream stream, spec_stream copy_stream,
                              void* const* layer_ready) {
  spec::Dims d;
  spec_status st = resolve(dm, &d);
  if (st != SPEC_OK) return st;
  if (!idx_now || !counts) return SPEC_ERR_INVALID;
  if (!aligned4(idx_now) || !aligned4(counts)) return SPEC_ERR_INVALID;
  if (copy_stream && !layer_ready) return SPEC_ERR_INVALID;
  if ((st = check_elastic(d, el)) != SPEC_OK) return st;
  if ((st = check_ws(d, SPEC_OP_DELTA, ws, ws_bytes)) != SPEC_OK) return st;
  HostKv hk;
  if ((st = resolve_host_kv(d, host, &hk)) != SPEC_OK) return st;
  const hipStream_t s = as_stream(stream);
  if (debug_on() && (st = debug_selection(d.B, d.k_max, 1, idx_now, counts, d.L_cap, s)) != SPEC_OK)
    return st;
  hipError_t e = spec::launch_delta_plan(d, idx_now, counts, el->slot_tok, el->slot_src,
                                         el->n_changed, ws, s);
  if (e != hipSuccess) return hip_status(e);
  st = enqueue_host_loads(d, hk, el, ws, d.n_layers, s, as_stream(copy_stream), layer_ready);
  if (st == SPEC_OK && debug_on() && copy_stream) st = finish(st, as_stream(copy_stream));
  return finish(st, s);
}

spec_status spec_step_offload(const spec_dims* dm, const uint16_t* q_r, const uint16_t* k_r,
                              const int32_t* seq_lens, const int32_t* ks, const uint16_t* q,
                              const uint16_t* k_cache, const uint16_t* v_cache,
                              int32_t n_dev_layers, const spec_host_kv* host, int32_t* idx_out,
                              int32_t* counts_out, float* out, float* lse, float* scores_out,
                              const spec_elastic* el, void* ws, size_t ws_bytes,
                              spec_stream stream, spec_stream copy_stream,
                              void* const* layer_ready) {
  spec::Dims d;
  spec_status st = resolve(dm, &d);
  if (st != SPEC_OK) return st;
  if (n_dev_layers < 0 || n_dev_layers >= d.n_layers) return SPEC_ERR_INVALID;
  if (!el) return SPEC_ERR_INVALID;
  // The device caches are needed only for device layers; the checks of
  // spec_step apply with stand-ins when there are none.
  const uint16_t* kc = n_dev_layers > 0 ? k_cache : q;
  const uint16_t* vc = n_dev_layers > 0 ? v_cache : q;
  if ((st = check_step(dm, &d, q_r, k_r, seq_lens, ks, q, kc, vc, idx_out, counts_out, out, lse,
                       scores_out, el)) != SPEC_OK)
    return st;
  if (copy_stream && !layer_ready) return SPEC_ERR_INVALID;
  if ((st = check_ws(d, SPEC_OP_OFFLOAD, ws, ws_bytes)) != SPEC_OK) return st;
  const int n_off = d.n_layers - n_dev_layers;
  spec::Dims d_off = d;   // the offloaded layers: the slot buffers and the host copy
  d_off.n_layers = n_off;
  HostKv hk;
  if ((st = resolve_host_kv(d_off, host, &hk)) != SPEC_OK) return st;
  const hipStream_t s = as_stream(stream);
  const hipStream_t cs = as_stream(copy_stream);
  if (debug_on() && (st = debug_lengths(d, seq_lens, ks, s)) != SPEC_OK) return st;

  char* p = static_cast<char*>(ws);
  float* scores = reinterpret_cast<float*>(p);
  p += spec::align_up(sizeof(float) * (size_t)d.B * d.n_sets * d.L_max);
  void* ws_score = p;
  p += spec::score_ws_bytes(d);
  void* ws_topk = p;
  p += spec::topk_ws_bytes(d);
  void* ws_attn = p;
  p += attn_ws_any_layers(d);
  void* ws_delta = p;

  hipError_t e = spec::launch_score_select(d, q_r, k_r, seq_lens, ks, scores_out, scores,
                                           idx_out, counts_out, ws_score, ws_topk, s);
  if (e != hipSuccess) return hip_status(e);
  e = spec::launch_delta_plan(d_off, idx_out, counts_out, el->slot_tok, el->slot_src,
                              el->n_changed, ws_delta,
                              s);
  if (e != hipSuccess) return hip_status(e);
  if ((st = enqueue_host_loads(d_off, hk, el, ws_delta, n_off, s, cs, layer_ready)) != SPEC_OK)
    return st;
  const size_t q_layer = (size_t)d.B * d.H_q * d.d;  // elements of q / out per layer
  if (n_dev_layers > 0) {  // the device layers, while the host rows are in flight
    spec::Dims d_dev = d;
    d_dev.n_layers = n_dev_layers;
    e = spec::launch_attn(d_dev, q, k_cache, v_cache, idx_out, counts_out, out, lse, ws_attn, s);
    if (e != hipSuccess) return hip_status(e);
  }
  spec::Dims d_one = d_off;  // one offloaded layer over its compact slots
  d_one.n_layers = 1;
  const int64_t slot_layer = (int64_t)d.B * d.k_max * d.H_kv * d.d;
  for (int l = 0; l < n_off; ++l) {
    if (cs && (e = hipStreamWaitEvent(s, static_cast<hipEvent_t>(layer_ready[l]), 0)) !=
                  hipSuccess)
      return hip_status(e);
    const size_t lo = (size_t)(n_dev_layers + l);
    e = spec::launch_attn(d_one, q + lo * q_layer, el->kbuf + l * slot_layer,
                          el->vbuf + l * slot_layer, nullptr, counts_out, out + lo * q_layer,
                          lse ? lse + lo * d.B * d.H_q : nullptr, ws_attn, s);
    if (e != hipSuccess) return hip_status(e);
  }
  return finish(SPEC_OK, s);
}

spec_status spec_retrieval_qk(const spec_dims* dm, const spec_frontend* fe,
                              const int32_t* tokens, const int32_t* pos, const uint16_t* emb,
                              const uint16_t* w_q, const uint16_t* w_k, uint16_t* q_r,
                              uint16_t* k_r, void* ws, size_t ws_bytes, spec_stream stream) {
  spec::Dims d;
  spec_status st = resolve(dm, &d);
  if (st != SPEC_OK) return st;
  spec::FrontDims f;
  if ((st = resolve_frontend(fe, &f)) != SPEC_OK) return st;
  if (!tokens || !pos || !emb || !w_q || !w_k || !q_r || !k_r) return SPEC_ERR_INVALID;
  if (!aligned4(tokens) || !aligned4(pos) || !aligned16(emb) || !aligned16(w_q) ||
      !aligned16(w_k) || !aligned16(q_r) || !aligned16(k_r))
    return SPEC_ERR_INVALID;
  if ((st = check_ws(d, SPEC_OP_FRONTEND, ws, ws_bytes)) != SPEC_OK) return st;
  if (debug_on()) {  // token ids the kernel would clamp into the table
    std::vector<int32_t> h;
    if (!d2h(h, tokens, (size_t)d.B, as_stream(stream))) return SPEC_ERR_HIP;
    for (int32_t v : h)
      if (v < 0 || v >= f.vocab) return SPEC_ERR_INVALID;
  }
  return finish(hip_status(spec::launch_retrieval_qk(d, f, tokens, pos, emb, w_q, w_k, q_r, k_r,
                                                     ws, as_stream(stream))),
                as_stream(stream));
}

const char* spec_status_string(spec_status s) {
  switch (s) {
    case SPEC_OK: return "ok";
    case SPEC_ERR_INVALID: return "invalid argument";
    case SPEC_ERR_UNSUPPORTED: return "unsupported dimensions";
    case SPEC_ERR_WORKSPACE: return "workspace missing or too small";
    case SPEC_ERR_HIP: return "HIP launch failed";
    case SPEC_ERR_TOO_LARGE:
      return "the step needs more workspace than the allocation-free entry point's static scratch";
  }
  return "unknown status";
}

int spec_last_hip_error(void) { return g_last_hip_error; }

const char* spec_version(void) { return "specctx 0.1.0 (gfx950)"; }

}  // extern "C"
