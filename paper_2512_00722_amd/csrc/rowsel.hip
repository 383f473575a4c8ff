// Retrieval scores and exact top-k of short sequences in one workgroup per
// score row (SpeContext Sec. 4.3: per-head softmax of the retrieval logits,
// Eq. 1, summed over the heads, then the k most important tokens).
//
// For a short sequence the tiled path (a softmax grid, then a classify grid
// and a select workgroup) is bound by its launches and round trips, not by
// its bytes (row_select_fits says which rows are short enough).  Here one
// 1024-thread workgroup per score row
//  * merges the logits kernel's per-block pairs into the head normalisers
//    (the same merge as the softmax kernel, so the scores are the same bits),
//  * forms the row's scores 4 tokens per thread (kept in the caller's buffer
//    only when asked for) and their order-preserving keys in LDS, with the
//    4096-bin histogram of the top 12 key bits,
//  * finds the k-th largest key T: the bin from that histogram, then two
//    10-bit LDS histogram passes over the keys of that bin,
//  * writes the selection in ascending token order: the keys above T and the
//    lowest-index r keys equal to T, placed by workgroup prefix sums over
//    the row in token order.
// A standalone selection (scores given) takes the same kernel from its second
// step on.
#include <stdlib.h>
#include <string.h>

#include "device_common.h"
#include "internal.h"
#include "score_norm.h"
#include "select_common.h"

namespace spec {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;

struct RowArgs {
  const float* logits;  // [B][H_r][L_max], log2 units; null: the scores are given
  const float* part;    // [B][H_r][n_blk][2] per-block (max, sum exp2)
  float* scores;        // [B * n_sets][L_max]: written from the logits (null: not kept), or read
  const int32_t* seq_lens;
  const int32_t* ks;
  int32_t* idx;     // [B * n_sets][k_max]
  int32_t* counts;  // [B] or null
  int L_max, k_max, H_r, n_sets, n_blk, tpb;
};

template <bool kFromLogits>
__global__ __launch_bounds__(kThreads) void row_select_kernel(RowArgs a) {
  __shared__ __align__(16) uint32_t s_key[kRowSelectMaxL];
  __shared__ int s_hist[kTopkBins];
  __shared__ int s_scan[2 * kWaves];
  __shared__ int s_sel[4];
  __shared__ float s_c[16];
  __shared__ float2 s_wred[4];

  const int srow = blockIdx.x;  // score row
  const int b = srow / a.n_sets;
  const int tid = threadIdx.x;
  const int L_raw = a.seq_lens[b];
  const int k_raw = a.ks[b];
  const int per = kFromLogits ? a.H_r / a.n_sets : 0;  // heads of this row
  const int h0 = (srow - b * a.n_sets) * per;
  HeadNorm nrm;
  if (kFromLogits) head_norm_load<true>(nrm, a.part, b, a.H_r, h0, per, a.n_blk);
  for (int i = tid; i < kTopkBins; i += kThreads) s_hist[i] = 0;
  if (tid == 0) s_sel[0] = s_sel[1] = s_sel[2] = -1;
  const int L_b = clampi(L_raw, 0, a.L_max);
  const int k_b = clampi(k_raw, 0, min(L_b, a.k_max));
  int32_t* out = a.idx + (size_t)srow * a.k_max;
  if (tid == 0 && a.counts && srow == b * a.n_sets) a.counts[b] = k_b;
  for (int j = k_b + tid; j < a.k_max; j += kThreads) out[j] = -1;

  if (kFromLogits) {
    head_norm_finish(nrm, (L_b + a.tpb - 1) / a.tpb, s_c, s_wred);  // ends with a barrier
    const bool sum_heads = a.n_sets == 1;
    const float* lg = a.logits + ((size_t)b * a.H_r + h0) * a.L_max;  // the row's first head
    float* keep = a.scores ? a.scores + (size_t)srow * a.L_max : nullptr;
    const bool vec = (a.L_max & 3) == 0;
    const bool vec_keep = vec && (reinterpret_cast<uintptr_t>(a.scores) & 15) == 0;
    for (int t0 = 4 * tid; t0 < a.L_max; t0 += 4 * kThreads) {
      float sc[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
      if (t0 < L_b) {
        float lv[4][16];
#pragma unroll
        for (int h = 0; h < 16; ++h) {
          if (h < per) {
            const float* l = lg + (size_t)h * a.L_max;
            if (vec && t0 + 3 < a.L_max) {
              const float4 v = *reinterpret_cast<const float4*>(l + t0);
              lv[0][h] = v.x;
              lv[1][h] = v.y;
              lv[2][h] = v.z;
              lv[3][h] = v.w;
            } else {  // row tail: clamped into the row; values past the length are unused
#pragma unroll
              for (int e = 0; e < 4; ++e) lv[e][h] = l[min(t0 + e, a.L_max - 1)];
            }
          }
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if (t0 + e < L_b) {
            float s = 0.f;
#pragma unroll
            for (int h = 0; h < 16; ++h)
              if (h < per) {
                const float w = exp2f(lv[e][h] - s_c[h]);
                s = sum_heads ? s + w : fmaxf(s, w);
              }
            sc[e] = s;
            const uint32_t key = order_key(s);
            s_key[t0 + e] = key;
            atomicAdd(&s_hist[key >> 20], 1);
          }
        }
      }
      if (keep) {
        if (vec_keep && t0 + 3 < a.L_max) {
          *reinterpret_cast<float4*>(keep + t0) = make_float4(sc[0], sc[1], sc[2], sc[3]);
        } else {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            if (t0 + e < a.L_max) keep[t0 + e] = sc[e];
        }
      }
    }
  } else {
    __syncthreads();  // the histogram is cleared
    const float* row = a.scores + (size_t)srow * a.L_max;
    for (int t0 = tid; t0 < L_b; t0 += 4 * kThreads) {
      float v[4];  // all four loads in flight, clamped into the sequence
#pragma unroll
      for (int u = 0; u < 4; ++u) v[u] = row[min(t0 + u * kThreads, L_b - 1)];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int t = t0 + u * kThreads;
        if (t < L_b) {
          const uint32_t key = order_key(v[u]);
          s_key[t] = key;
          atomicAdd(&s_hist[key >> 20], 1);
        }
      }
    }
  }
  __syncthreads();
  if (k_b == 0 || k_b == L_b) {  // nothing, or every token, is selected
    for (int j = tid; j < k_b; j += kThreads) out[j] = j;
    return;
  }

  // ---- the k-th largest key T: top 12 bits, then 10 + 10 bits
  find_bin<kThreads>(s_hist, kTopkBins, k_b, s_scan, s_sel);
  uint32_t T = (uint32_t)s_sel[0] << 20;
  int remaining = k_b - s_sel[1];  // keys still to take at or below T's prefix
#pragma unroll 1
  for (int pass = 0; pass < 2; ++pass) {
    const int shift = pass == 0 ? 10 : 0;
    const uint32_t hi_mask = pass == 0 ? 0xFFF00000u : 0xFFFFFC00u;
    __syncthreads();  // every thread has read s_sel and s_hist
    for (int i = tid; i < 1024; i += kThreads) s_hist[i] = 0;
    __syncthreads();
    for (int t = tid; t < L_b; t += kThreads) {
      const uint32_t kk = s_key[t];
      if ((kk & hi_mask) == T) atomicAdd(&s_hist[(kk >> shift) & 1023], 1);
    }
    __syncthreads();
    find_bin<kThreads>(s_hist, 1024, remaining, s_scan, s_sel);
    T |= (uint32_t)s_sel[0] << shift;
    remaining -= s_sel[1];
  }
  const int r = remaining;  // keys equal to T to take, lowest index first

  // ---- ordered compaction: 4 consecutive tokens per thread and round
  int carry_gt = 0, carry_eq = 0;
  for (int base = 0; base < L_b; base += 4 * kThreads) {
    const int t0 = base + 4 * tid;
    uint32_t key[4] = {0u, 0u, 0u, 0u};
    if (t0 < L_b) {  // t0 + 3 < kRowSelectMaxL: t0 is a multiple of 4 below it
      const uint4 k4 = *reinterpret_cast<const uint4*>(&s_key[t0]);
      key[0] = k4.x;
      key[1] = k4.y;
      key[2] = k4.z;
      key[3] = k4.w;
    }
    int ngt = 0, neq = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const bool valid = t0 + e < L_b;
      ngt += valid && key[e] > T;
      neq += valid && key[e] == T;
    }
    int gt_before, eq_before, gt_tot, eq_tot;
    block_scan2<kThreads>(ngt, neq, gt_before, eq_before, gt_tot, eq_tot, s_scan);
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

bool force_tiles() {
  const char* p = getenv("SPEC_TOPK_PATH");
  return p && strcmp(p, "tiles") == 0;
}

}  // namespace

bool row_select_fits(const Dims& d, int heads_per_row) {
  return d.L_max <= kRowSelectMaxL &&
         (int64_t)heads_per_row * d.L_max <= kRowSelectMaxLogits && !force_tiles();
}

hipError_t launch_row_select(const Dims& d, void* ws_score, float* scores,
                             const int32_t* seq_lens, const int32_t* ks, int32_t* idx,
                             int32_t* counts, hipStream_t s) {
  RowArgs a{ws_score ? score_ws_logits(ws_score) : nullptr,
            ws_score ? score_ws_part(d, ws_score) : nullptr,
            scores, seq_lens, ks, idx, counts, d.L_max, d.k_max, d.H_r, d.n_sets,
            score_blocks(d), score_tokens_per_block(d)};
  const dim3 grid((unsigned)(d.B * d.n_sets));
  if (ws_score)
    row_select_kernel<true><<<grid, kThreads, 0, s>>>(a);
  else
    row_select_kernel<false><<<grid, kThreads, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_score_select(const Dims& d, const uint16_t* q_r, const uint16_t* k_r,
                               const int32_t* seq_lens, const int32_t* ks, float* scores_keep,
                               float* scores_ws, int32_t* idx, int32_t* counts, void* ws_score,
                               void* ws_topk, hipStream_t s) {
  if (row_select_fits(d, d.H_r / d.n_sets)) {
    hipError_t e = launch_logits(d, q_r, k_r, seq_lens, ws_score, false, s);
    if (e != hipSuccess) return e;
    return launch_row_select(d, ws_score, scores_keep, seq_lens, ks, idx, counts, s);
  }
  float* scores = scores_keep ? scores_keep : scores_ws;
  hipError_t e = launch_score(d, q_r, k_r, seq_lens, scores, ws_score, s);
  if (e != hipSuccess) return e;
  // The score kernels already built the selection histogram.
  return launch_topk_select(d, scores, seq_lens, ks, score_ws_hist(d, ws_score),
                            static_cast<char*>(ws_topk) + topk_hist_bytes(d), idx, counts, s);
}

}  // namespace spec
