// Exact top-k token selection on gfx950 (SpeContext Sec. 4.3: the important
// tokens are chosen from the retrieval head's attention weights).
//
// One 1024-thread workgroup per sequence.  The fp32 scores are mapped to
// order-preserving 32-bit keys and the k-th largest key T is found by a
// radix select over three digits (bits 31..20, 19..8, 7..0) with LDS
// histograms; only keys that share the digits chosen so far are counted in
// later passes.  The select also yields r, the number of keys equal to T that
// belong to the set (the lowest-index ones: ties go to the lower index).
// A final ordered compaction walks the row in index order; one workgroup
// scan of the pair (#keys > T, #keys == T) gives every selected token its
// output slot, so the indices come out ascending with no sort.
#include "device_common.h"
#include "internal.h"

namespace spec {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;

struct TopkArgs {
  const float* scores;  // [B][L_max]
  const int32_t* seq_lens;
  const int32_t* ks;
  int32_t* idx;         // [B][k_max]
  int32_t* counts;      // [B] or null
  int L_max, k_max;
};

// Exclusive scan of two ints over the workgroup; returns the totals too.
// Must be called by all threads.
__device__ __forceinline__ void block_scan2(int a, int b, int& ea, int& eb, int& ta, int& tb,
                                            int* sh /* [2*kWaves + 2] */) {
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  int ia = a, ib = b;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int na = __shfl_up(ia, off);
    const int nb = __shfl_up(ib, off);
    if (lane >= off) {
      ia += na;
      ib += nb;
    }
  }
  if (lane == 63) {
    sh[wave] = ia;
    sh[kWaves + wave] = ib;
  }
  __syncthreads();
  if (wave == 0) {
    int wa = lane < kWaves ? sh[lane] : 0;
    int wb = lane < kWaves ? sh[kWaves + lane] : 0;
#pragma unroll
    for (int off = 1; off < kWaves; off <<= 1) {
      const int na = __shfl_up(wa, off);
      const int nb = __shfl_up(wb, off);
      if (lane >= off) {
        wa += na;
        wb += nb;
      }
    }
    if (lane < kWaves) {
      sh[lane] = wa;  // inclusive prefix over waves
      sh[kWaves + lane] = wb;
    }
  }
  __syncthreads();
  const int pa = wave > 0 ? sh[wave - 1] : 0;
  const int pb = wave > 0 ? sh[kWaves + wave - 1] : 0;
  ea = pa + ia - a;
  eb = pb + ib - b;
  ta = sh[kWaves - 1];
  tb = sh[2 * kWaves - 1];
  __syncthreads();  // sh is reused by the next call
}

__global__ __launch_bounds__(kThreads) void topk_kernel(TopkArgs a) {
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int L_b = clampi(a.seq_lens[b], 0, a.L_max);
  const int k_b = clampi(a.ks[b], 0, min(L_b, a.k_max));
  const float* row = a.scores + (size_t)b * a.L_max;
  int32_t* out = a.idx + (size_t)b * a.k_max;

  if (tid == 0 && a.counts) a.counts[b] = k_b;
  for (int j = k_b + tid; j < a.k_max; j += kThreads) out[j] = -1;
  if (k_b == 0 || k_b == L_b) {  // nothing, or every token, is selected
    for (int j = tid; j < k_b; j += kThreads) out[j] = j;
    return;
  }

  __shared__ int hist[4096];
  __shared__ int scan_sh[2 * kWaves + 2];
  __shared__ int sel_digit, sel_above;

  uint32_t prefix = 0, mask = 0;
  int remaining = k_b;  // keys still to take at or below the current prefix
#pragma unroll 1
  for (int pass = 0; pass < 3; ++pass) {
    const int shift = pass == 0 ? 20 : (pass == 1 ? 8 : 0);
    const int nbins = pass < 2 ? 4096 : 256;
    for (int i = tid; i < nbins; i += kThreads) hist[i] = 0;
    __syncthreads();
    for (int t = tid; t < L_b; t += kThreads) {
      const uint32_t key = order_key(row[t]);
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & (nbins - 1)], 1);
    }
    __syncthreads();
    // Thread i owns bins in descending order: digits nbins-1-i*bpt ... .
    const int bpt = nbins >= kThreads ? nbins / kThreads : 1;
    const bool owns = tid * bpt < nbins;
    int cnt[4] = {0, 0, 0, 0};
    int local = 0;
    if (owns) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (e < bpt) {
          cnt[e] = hist[nbins - 1 - (tid * bpt + e)];
          local += cnt[e];
        }
      }
    }
    int before, dummy, tot, tot2;
    block_scan2(local, 0, before, dummy, tot, tot2, scan_sh);
    if (owns) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if (e >= bpt) break;
        if (before < remaining && remaining <= before + cnt[e]) {
          sel_digit = nbins - 1 - (tid * bpt + e);
          sel_above = before;
        }
        before += cnt[e];
      }
    }
    __syncthreads();
    prefix |= (uint32_t)sel_digit << shift;
    mask |= (uint32_t)(nbins - 1) << shift;
    remaining -= sel_above;
    __syncthreads();  // sel_* are rewritten by the next pass
  }
  const uint32_t T = prefix;  // key of the k_b-th largest score
  const int r = remaining;    // keys equal to T that are taken (lowest indices)

  // Ordered compaction: thread tid covers 4 consecutive tokens per chunk.
  int carry_gt = 0, carry_eq = 0;
  for (int base = 0; base < L_b; base += 4 * kThreads) {
    const int t0 = base + 4 * tid;
    uint32_t key[4];
    int ngt = 0, neq = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      key[e] = (t0 + e < L_b) ? order_key(row[t0 + e]) : 0u;
      const bool valid = t0 + e < L_b;
      ngt += (valid && key[e] > T);
      neq += (valid && key[e] == T);
    }
    int gt_before, eq_before, gt_tot, eq_tot;
    block_scan2(ngt, neq, gt_before, eq_before, gt_tot, eq_tot, scan_sh);
    gt_before += carry_gt;
    eq_before += carry_eq;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      if (t0 + e >= L_b) break;
      if (key[e] > T) {
        out[gt_before + min(eq_before, r)] = t0 + e;
        ++gt_before;
      } else if (key[e] == T) {
        if (eq_before < r) out[gt_before + eq_before] = t0 + e;
        ++eq_before;
      }
    }
    carry_gt += gt_tot;
    carry_eq += eq_tot;
  }
}

}  // namespace

hipError_t launch_topk(const Dims& d, const float* scores, const int32_t* seq_lens,
                       const int32_t* ks, int32_t* idx, int32_t* counts, void* /*ws*/,
                       hipStream_t s) {
  TopkArgs a{scores, seq_lens, ks, idx, counts, d.L_max, d.k_max};
  topk_kernel<<<d.B, kThreads, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace spec
