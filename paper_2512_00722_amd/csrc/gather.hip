// KV row movement on gfx950: the materialised gather of the selected rows
// (SpeContext Sec. 4.3 "Support for MHA": the selected KV is loaded per head)
// and elastic loading (Sec. 5.4: keep S_last on the device, load only
// S_now - S_last into the places freed by S_last - S_now).
//
// A token's K (or V) row of one layer is H_kv*d bf16 = 2 KiB contiguous in
// the token-major cache, so every copy is whole rows moved with 16-byte
// lanes: 128 lanes per row, fully coalesced on both sides.
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
  int B, k_max, L_cap;
};

// grid (ceil(k_max / 16), B, n_layers)
__global__ __launch_bounds__(256) void gather_kernel(GatherArgs a) {
  const int b = blockIdx.y;
  const int layer = blockIdx.z;
  const int count = clampi(a.counts[b], 0, a.k_max);
  const int j0 = blockIdx.x * kRowsPerBlock;
  if (j0 >= count) return;
  const int nrows = min(kRowsPerBlock, count - j0);
  const int cpr = (int)(a.row_elems / 8);  // 16-byte chunks per row
  const uint16_t* ks = a.k + (int64_t)layer * a.stride_layer + (int64_t)b * a.stride_b;
  const uint16_t* vs = a.v + (int64_t)layer * a.stride_layer + (int64_t)b * a.stride_b;
  const int64_t dst0 = ((int64_t)layer * a.B + b) * a.k_max * a.row_elems;
  for (int x = threadIdx.x; x < nrows * cpr; x += 256) {
    const int r = x / cpr;
    const int c = x - r * cpr;
    const int j = j0 + r;
    const int tok = clampi(a.idx[(size_t)b * a.k_max + j], 0, a.L_cap - 1);
    const int64_t src = (int64_t)tok * a.row_elems + 8 * c;
    const int64_t dst = dst0 + (int64_t)j * a.row_elems + 8 * c;
    *reinterpret_cast<uint4*>(a.k_sel + dst) = ldg16(ks + src);
    *reinterpret_cast<uint4*>(a.v_sel + dst) = ldg16(vs + src);
  }
}

// ---------------------------------------------------------------- elastic

constexpr int kPlanThreads = 1024;
constexpr int kPlanWaves = kPlanThreads / 64;

struct PlanArgs {
  const int32_t* idx_now;  // [B][k_max], S_now = idx_now[b][0..counts[b]) ascending
  const int32_t* counts;
  int32_t* slot_tok;       // [B][k_max]
  int32_t* n_changed;      // [B]
  int32_t* loads;          // ws: [B][k_max][2] (slot, token)
  int k_max, L_cap;
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
  for (int i = tid; i < n_apply; i += kPlanThreads) slot[loads[2 * i]] = loads[2 * i + 1];
  if (tid == 0) a.n_changed[b] = n_apply;
}

struct CopyArgs {
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* loads;
  const int32_t* n_changed;
  uint16_t* kbuf;
  uint16_t* vbuf;
  int64_t stride_layer, stride_b, row_elems;
  int B, k_max, L_cap;
};

// grid (ceil(k_max / 16), B, n_layers): copy the loaded rows into their slots.
__global__ __launch_bounds__(256) void elastic_copy_kernel(CopyArgs a) {
  const int b = blockIdx.y;
  const int layer = blockIdx.z;
  const int n = clampi(a.n_changed[b], 0, a.k_max);
  const int i0 = blockIdx.x * kRowsPerBlock;
  if (i0 >= n) return;
  const int nrows = min(kRowsPerBlock, n - i0);
  const int cpr = (int)(a.row_elems / 8);
  const int32_t* loads = a.loads + (size_t)b * a.k_max * 2;
  const uint16_t* ks = a.k + (int64_t)layer * a.stride_layer + (int64_t)b * a.stride_b;
  const uint16_t* vs = a.v + (int64_t)layer * a.stride_layer + (int64_t)b * a.stride_b;
  const int64_t dst0 = ((int64_t)layer * a.B + b) * a.k_max * a.row_elems;
  for (int x = threadIdx.x; x < nrows * cpr; x += 256) {
    const int r = x / cpr;
    const int c = x - r * cpr;
    const int i = i0 + r;
    const int slot = clampi(loads[2 * i], 0, a.k_max - 1);
    const int tok = clampi(loads[2 * i + 1], 0, a.L_cap - 1);
    const int64_t src = (int64_t)tok * a.row_elems + 8 * c;
    const int64_t dst = dst0 + (int64_t)slot * a.row_elems + 8 * c;
    *reinterpret_cast<uint4*>(a.kbuf + dst) = ldg16(ks + src);
    *reinterpret_cast<uint4*>(a.vbuf + dst) = ldg16(vs + src);
  }
}

}  // namespace

hipError_t launch_gather(const Dims& d, const uint16_t* k_cache, const uint16_t* v_cache,
                         const int32_t* idx, const int32_t* counts, uint16_t* k_sel,
                         uint16_t* v_sel, hipStream_t s) {
  GatherArgs a{k_cache, v_cache, idx, counts, k_sel, v_sel, d.kv_stride_layer, d.kv_stride_b,
               (int64_t)d.H_kv * d.d, d.B, d.k_max, d.L_cap};
  const dim3 grid((d.k_max + kRowsPerBlock - 1) / kRowsPerBlock, d.B, d.n_layers);
  gather_kernel<<<grid, 256, 0, s>>>(a);
  return hipGetLastError();
}

size_t elastic_plan_lds_bytes(const Dims& d) {
  return sizeof(uint32_t) * 2 * (size_t)((d.L_cap + 31) / 32);
}

hipError_t launch_delta(const Dims& d, const int32_t* idx_now, const int32_t* counts,
                        const uint16_t* k_cache, const uint16_t* v_cache,
                        int32_t* slot_tok, uint16_t* kbuf, uint16_t* vbuf,
                        int32_t* n_changed, void* ws, hipStream_t s) {
  int32_t* loads = static_cast<int32_t*>(ws);
  PlanArgs p{idx_now, counts, slot_tok, n_changed, loads, d.k_max, d.L_cap};
  elastic_plan_kernel<<<d.B, kPlanThreads, elastic_plan_lds_bytes(d), s>>>(p);
  CopyArgs c{k_cache, v_cache, loads, n_changed, kbuf, vbuf, d.kv_stride_layer, d.kv_stride_b,
             (int64_t)d.H_kv * d.d, d.B, d.k_max, d.L_cap};
  const dim3 grid((d.k_max + kRowsPerBlock - 1) / kRowsPerBlock, d.B, d.n_layers);
  elastic_copy_kernel<<<grid, 256, 0, s>>>(c);
  return hipGetLastError();
}

}  // namespace spec
