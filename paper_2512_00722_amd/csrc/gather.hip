// KV row movement on gfx950: the materialised gather of the selected rows
// (SpeContext Sec. 4.3 "Support for MHA": the selected KV is loaded per head)
// and elastic loading (Sec. 5.4: keep S_last on the device, load only
// S_now - S_last into the places freed by S_last - S_now).
//
// A token's K (or V) row of one layer is H_kv*d bf16 contiguous in the
// token-major cache (2 KiB at H_kv = 8), so every copy is whole rows moved
// with 16-byte lanes (128 lanes per 2 KiB row), fully coalesced on both sides.
#include "device_common.h"
#include "internal.h"

namespace spec {
namespace {

constexpr int kRowsPerBlock = 16;

struct GatherArgs {
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* idx;     // [B][k_max]
  const int32_t* counts;  // [B]
  uint16_t* k_sel;        // [n_layers][B][k_max][H_kv][d]
  uint16_t* v_sel;
  int64_t stride_layer, stride_b, row_elems;
  int B, k_max, L_cap, n_layers, n_sets;
};

// 16-byte store that bypasses cache retention (the rows are consumed later,
// by another launch, and exceed the caches anyway).
__device__ __forceinline__ void stg16_stream(uint16_t* p, const uint4& v) {
  uint4* q = reinterpret_cast<uint4*>(p);
  __builtin_nontemporal_store(v.x, &q->x);
  __builtin_nontemporal_store(v.y, &q->y);
  __builtin_nontemporal_store(v.z, &q->z);
  __builtin_nontemporal_store(v.w, &q->w);
}

// Copies of whole rows.  The block's (source row, destination row) pairs are
// staged in LDS first (one index round trip), then every lane issues all its
// loads (kCopyUnroll K and V chunks) before its first store, so each lane
// keeps 2*kCopyUnroll 16-byte loads in flight.
constexpr int kCopyUnroll = 8;

// src_row holds `nsrc` source rows per destination row: one (the row moves
// whole) or one per KV head (head h's cph chunks come from its own row).
__device__ __forceinline__ void copy_rows(const uint16_t* __restrict__ ks,
                                          const uint16_t* __restrict__ vs,
                                          uint16_t* __restrict__ kd, uint16_t* __restrict__ vd,
                                          int nrows, int cpr, int64_t row_elems,
                                          const int64_t* src_row, const int64_t* dst_row,
                                          int nsrc = 1, int cph = 1) {
  const int total = nrows * cpr;
  for (int x0 = threadIdx.x; x0 < total; x0 += 256 * kCopyUnroll) {
    uint4 kr[kCopyUnroll], vr[kCopyUnroll];
    int64_t dst[kCopyUnroll];
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
      const int x = x0 + 256 * u;
      dst[u] = -1;
      if (x < total) {
        const int r = x / cpr;
        const int c = x - r * cpr;
        const int64_t src = src_row[r * nsrc + (nsrc > 1 ? c / cph : 0)] * row_elems + 8 * c;
        dst[u] = dst_row[r] * row_elems + 8 * c;
        kr[u] = ldg16_stream(ks + src);
        vr[u] = ldg16_stream(vs + src);
      }
    }
#pragma unroll
    for (int u = 0; u < kCopyUnroll; ++u) {
      if (dst[u] >= 0) {
        stg16_stream(kd + dst[u], kr[u]);
        stg16_stream(vd + dst[u], vr[u]);
      }
    }
  }
}

// grid (ceil(k_max / 16), B): 16 selected rows of one sequence, every layer.
// With one token set per KV head (n_sets = H_kv), row j of the output holds,
// for each head g, the head-g piece of token idx[b][g][j].
__global__ __launch_bounds__(256) void gather_kernel(GatherArgs a) {
  const int b = blockIdx.y;
  const int count = clampi(a.counts[b], 0, a.k_max);
  const int j0 = blockIdx.x * kRowsPerBlock;
  if (j0 >= count) return;
  const int nrows = min(kRowsPerBlock, count - j0);
  const int cpr = (int)(a.row_elems / 8);  // 16-byte chunks per row
  const int ns = a.n_sets;                 // source rows per output row
  __shared__ int64_t src_row[kRowsPerBlock * 16], dst_row[kRowsPerBlock];
  for (int e = threadIdx.x; e < nrows * ns; e += 256) {
    const int r = e / ns, g = e - r * ns;
    src_row[e] = clampi(a.idx[((size_t)b * ns + g) * a.k_max + j0 + r], 0, a.L_cap - 1);
  }
  if (threadIdx.x < nrows) dst_row[threadIdx.x] = (int64_t)b * a.k_max + j0 + threadIdx.x;
  __syncthreads();
  const int64_t layer_rows = (int64_t)a.B * a.k_max;  // rows per layer of the output
  for (int layer = 0; layer < a.n_layers; ++layer) {
    const int64_t off = (int64_t)layer * a.stride_layer + (int64_t)b * a.stride_b;
    const int64_t doff = layer * layer_rows * a.row_elems;
    copy_rows(a.k + off, a.v + off, a.k_sel + doff, a.v_sel + doff, nrows, cpr, a.row_elems,
              src_row, dst_row, ns, cpr / (ns > 1 ? ns : 1));
  }
}

// ---------------------------------------------------------------- elastic

constexpr int kPlanThreads = 1024;
constexpr int kPlanWaves = kPlanThreads / 64;

struct PlanArgs {
  const int32_t* idx_now;  // [B][k_max], S_now = idx_now[b][0..counts[b]) ascending
  const int32_t* counts;
  int32_t* slot_tok;       // [B][k_max]
  int32_t* slot_src;       // [B][k_max]: token loaded into the slot by this update, or -1
  int32_t* n_changed;      // [B]
  int32_t* loads;          // ws: [B][k_max][2] (slot, token)
  int32_t* fused;          // ws: [B] 1: the attention loads this sequence's rows (or null)
  int k_max, L_cap;
  int fuse_pct;            // fused when more than fuse_pct % of the selection is new
};

// Exclusive workgroup scan of one int; returns the total.
__device__ __forceinline__ int plan_scan(int x, int& total, int* sh) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  int inc = x;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int n = __shfl_up(inc, off);
    if (lane >= off) inc += n;
  }
  if (lane == 63) sh[wave] = inc;
  __syncthreads();
  if (wave == 0) {
    int w = lane < kPlanWaves ? sh[lane] : 0;
#pragma unroll
    for (int off = 1; off < kPlanWaves; off <<= 1) {
      const int n = __shfl_up(w, off);
      if (lane >= off) w += n;
    }
    if (lane < kPlanWaves) sh[lane] = w;
  }
  __syncthreads();
  const int ex = (wave > 0 ? sh[wave - 1] : 0) + inc - x;
  total = sh[kPlanWaves - 1];
  __syncthreads();
  return ex;
}

// One workgroup per sequence: set differences and the slot assignment.
// Dynamic LDS: two bitmaps over L_cap tokens (S_now, and S_now held already).
__global__ __launch_bounds__(kPlanThreads) void elastic_plan_kernel(PlanArgs a) {
  extern __shared__ uint32_t bits[];
  __shared__ int sh[kPlanWaves + 2];
  __shared__ int any_high;
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int words = (a.L_cap + 31) / 32;
  uint32_t* now_bits = bits;
  uint32_t* held_bits = bits + words;
  const int c = clampi(a.counts[b], 0, a.k_max);
  const int32_t* s_now = a.idx_now + (size_t)b * a.k_max;
  int32_t* slot = a.slot_tok + (size_t)b * a.k_max;
  int32_t* src = a.slot_src + (size_t)b * a.k_max;
  int32_t* loads = a.loads + (size_t)b * a.k_max * 2;

  for (int w = tid; w < 2 * words; w += kPlanThreads) bits[w] = 0u;
  if (tid == 0) any_high = 0;
  __syncthreads();
  for (int j = tid; j < c; j += kPlanThreads) {
    const int t = s_now[j];
    if (t >= 0 && t < a.L_cap) atomicOr(&now_bits[t >> 5], 1u << (t & 31));
  }
  __syncthreads();
  // A slot is kept if its token is in S_now.  A kept slot at or beyond c
  // (the budget shrank) breaks the "slots [0, c) hold S_now" layout: then
  // this sequence is reloaded in full.
  for (int s = tid; s < a.k_max; s += kPlanThreads) {
    const int t = slot[s];
    const bool keep = t >= 0 && t < a.L_cap && ((now_bits[t >> 5] >> (t & 31)) & 1u);
    if (keep && s >= c) any_high = 1;
  }
  __syncthreads();
  const bool full = any_high != 0;
  for (int s = tid; s < a.k_max; s += kPlanThreads) {
    const int t = slot[s];
    const bool keep = !full && t >= 0 && t < a.L_cap && ((now_bits[t >> 5] >> (t & 31)) & 1u);
    if (keep) atomicOr(&held_bits[t >> 5], 1u << (t & 31));
  }
  __syncthreads();

  // D_in = S_now - S_last in ascending token order (S_now is ascending):
  // its i-th element goes to the i-th free slot in ascending slot order.
  int n_in_total = 0;
  int base_in = 0;
  for (int j0 = 0; j0 < c; j0 += kPlanThreads) {
    const int j = j0 + tid;
    int t = -1;
    int is_in = 0;
    if (j < c) {
      t = s_now[j];
      is_in = (t >= 0 && t < a.L_cap) ? !((held_bits[t >> 5] >> (t & 31)) & 1u) : 0;
    }
    int tot;
    const int pos = plan_scan(is_in, tot, sh) + base_in;
    if (is_in) loads[2 * pos + 1] = t;
    base_in += tot;
  }
  n_in_total = base_in;

  // Free slots in ascending order: the first n_in receive D_in, the rest
  // become empty.  Each slot is read and written by one thread only here.
  int base_free = 0;
  for (int s0 = 0; s0 < a.k_max; s0 += kPlanThreads) {
    const int s = s0 + tid;
    int is_free = 0;
    if (s < a.k_max) {
      const int t = slot[s];
      const bool keep = !full && t >= 0 && t < a.L_cap && ((now_bits[t >> 5] >> (t & 31)) & 1u);
      is_free = !keep;
      src[s] = -1;  // loaded slots are set below, after the barrier
    }
    int tot;
    const int pos = plan_scan(is_free, tot, sh) + base_free;
    if (is_free) {
      if (pos < n_in_total)
        loads[2 * pos] = s;
      else
        slot[s] = -1;
    }
    base_free += tot;
  }
  // A consistent state (distinct slot tokens) always has enough free slots;
  // a corrupted one must still never index outside the slot row.
  const int n_apply = min(n_in_total, base_free);
  __syncthreads();  // loads[] complete before it is applied
  for (int i = tid; i < n_apply; i += kPlanThreads) {
    slot[loads[2 * i]] = loads[2 * i + 1];
    src[loads[2 * i]] = loads[2 * i + 1];
  }
  if (tid == 0) {
    a.n_changed[b] = n_apply;
    if (a.fused) a.fused[b] = (int64_t)100 * n_apply > (int64_t)a.fuse_pct * c ? 1 : 0;
  }
}

struct CopyArgs {
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* loads;
  const int32_t* n_changed;
  const int32_t* skip;      // [B] or null: sequences whose rows the attention loads
  uint16_t* kbuf;
  uint16_t* vbuf;
  int64_t stride_layer, stride_b, row_elems;
  int B, k_max, L_cap, n_layers;
};

// grid (ceil(k_max / 16), B): copy 16 loaded rows of one sequence into their
// slots, every layer.
__global__ __launch_bounds__(256) void elastic_copy_kernel(CopyArgs a) {
  const int b = blockIdx.y;
  const int n = a.skip && a.skip[b] ? 0 : clampi(a.n_changed[b], 0, a.k_max);
  const int i0 = blockIdx.x * kRowsPerBlock;
  if (i0 >= n) return;
  const int nrows = min(kRowsPerBlock, n - i0);
  const int cpr = (int)(a.row_elems / 8);
  __shared__ int64_t src_row[kRowsPerBlock], dst_row[kRowsPerBlock];
  if (threadIdx.x < nrows) {
    const int32_t* ld = a.loads + ((size_t)b * a.k_max + i0 + threadIdx.x) * 2;
    dst_row[threadIdx.x] = (int64_t)b * a.k_max + clampi(ld[0], 0, a.k_max - 1);
    src_row[threadIdx.x] = clampi(ld[1], 0, a.L_cap - 1);
  }
  __syncthreads();
  const int64_t layer_rows = (int64_t)a.B * a.k_max;
  for (int layer = 0; layer < a.n_layers; ++layer) {
    const int64_t off = (int64_t)layer * a.stride_layer + (int64_t)b * a.stride_b;
    const int64_t doff = layer * layer_rows * a.row_elems;
    copy_rows(a.k + off, a.v + off, a.kbuf + doff, a.vbuf + doff, nrows, cpr, a.row_elems,
              src_row, dst_row);
  }
}

}  // namespace

// The elastic copy, device to device, runs at most kCopyPerCU workgroups per
// CU (dynamic LDS is reserved for the purpose; registers would allow five):
// on 64 ragged sequences whose steady updates read and write 2.75 GB, whole
// steps went from 3622 to 3439 us with two per CU (one and three: within 1%
// of two).  Copies from host memory keep every workgroup the CU holds: the
// host link's latency needs their requests in flight.  The materialised
// gather keeps full occupancy too (the cap made it slower).
constexpr int kCopyPerCU = 2;
constexpr size_t kCopyLdsPerCU = 160 * 1024;

hipError_t launch_gather(const Dims& d, const uint16_t* k_cache, const uint16_t* v_cache,
                         const int32_t* idx, const int32_t* counts, uint16_t* k_sel,
                         uint16_t* v_sel, hipStream_t s) {
  GatherArgs a{k_cache, v_cache, idx, counts, k_sel, v_sel, d.kv_stride_layer, d.kv_stride_b,
               (int64_t)d.H_kv * d.d, d.B, d.k_max, d.L_cap, d.n_layers, d.n_sets};
  const dim3 grid((d.k_max + kRowsPerBlock - 1) / kRowsPerBlock, d.B);
  gather_kernel<<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

size_t elastic_plan_lds_bytes(const Dims& d) {
  return sizeof(uint32_t) * 2 * (size_t)((d.L_cap + 31) / 32);
}

hipError_t launch_delta_plan(const Dims& d, const int32_t* idx_now, const int32_t* counts,
                             int32_t* slot_tok, int32_t* slot_src, int32_t* n_changed, void* ws,
                             hipStream_t s, int fuse_pct) {
  PlanArgs p{idx_now, counts, slot_tok, slot_src, n_changed, static_cast<int32_t*>(ws),
             fuse_pct >= 0 ? delta_ws_fused(d, ws) : nullptr, d.k_max, d.L_cap, fuse_pct};
  elastic_plan_kernel<<<d.B, kPlanThreads, elastic_plan_lds_bytes(d), s>>>(p);
  return hipGetLastError();
}

hipError_t launch_delta_copy(const Dims& d, const uint16_t* k_src, const uint16_t* v_src,
                             int64_t src_stride_layer, int64_t src_stride_b, int n_layers,
                             const int32_t* n_changed, uint16_t* kbuf, uint16_t* vbuf,
                             const void* ws, hipStream_t s, const int32_t* skip, bool from_host) {
  CopyArgs c{k_src, v_src, static_cast<const int32_t*>(ws), n_changed, skip, kbuf, vbuf,
             src_stride_layer, src_stride_b, (int64_t)d.H_kv * d.d, d.B, d.k_max, d.L_cap,
             n_layers};
  const dim3 grid((d.k_max + kRowsPerBlock - 1) / kRowsPerBlock, d.B);
  const size_t lds = from_host ? 0 : kCopyLdsPerCU / kCopyPerCU - 4096;  // two fit, three do not
  elastic_copy_kernel<<<grid, 256, lds, s>>>(c);
  return hipGetLastError();
}

hipError_t launch_delta(const Dims& d, const int32_t* idx_now, const int32_t* counts,
                        const uint16_t* k_cache, const uint16_t* v_cache,
                        int32_t* slot_tok, int32_t* slot_src, uint16_t* kbuf, uint16_t* vbuf,
                        int32_t* n_changed, void* ws, hipStream_t s) {
  hipError_t e = launch_delta_plan(d, idx_now, counts, slot_tok, slot_src, n_changed, ws, s);
  if (e != hipSuccess) return e;
  return launch_delta_copy(d, k_cache, v_cache, d.kv_stride_layer, d.kv_stride_b, d.n_layers,
                           n_changed, kbuf, vbuf, ws, s);
}

}  // namespace spec
