// Retrieval scoring on gfx950 (SpeContext Sec. 4.3; Eq. 1 per retrieval head,
// then the sum over heads of Sec. 4.2's batch-level mapping).
//
// Two launches:
//  1. logits_kernel streams K_r once.  Each lane holds 8 bf16 of one
//     (token, head) row slice in one 16-byte load; the d_r/8 lanes of a head
//     reduce their partial dot products with cross-lane shuffles.  A
//     workgroup covers 256 tokens (64 or 128 when the grid would not cover
//     the CUs); it writes the logits (log2 units, the scale and log2(e)
//     folded into q_r) and its per-head (max, sum exp2).
//  2. softmax_headsum_kernel merges the per-block pairs into each head's
//     normaliser c_h = M_h + log2 Z_h and writes
//     score[t] = sum_h exp2(l[h,t] - c_h), -inf beyond the sequence length.
// The softmax needs every head's global max and sum before any score can be
// formed, hence the logits round trip (1/(d_r/2) of the K_r bytes).
#include "device_common.h"
#include "internal.h"
#include "score_norm.h"

namespace spec {
namespace {

constexpr int T2 = kSoftTokensPerBlock;
// Rows in flight per lane: 4 where the grid covers the CUs several times
// over (more would only lengthen the queues), 8 for small grids, whose few
// workgroups must each keep more bytes in flight.
constexpr int kUnrollWide = 4;
constexpr int kUnrollNarrow = 8;

struct LogitsArgs {
  const uint16_t* q_r;
  const uint16_t* k_r;
  const int32_t* seq_lens;
  float* logits;  // [B][H_r][L_max], log2 units
  float* part;    // [B][H_r][n_blk][2]: block max, block sum of exp2(l - max)
  int32_t* hist;  // [B][n_sets][4096] top-k histograms, zeroed here for the next kernel (or null)
  int64_t kr_stride_b;
  int L_max, H_r, n_blk, n_sets;
  float qscale;   // scale_r * log2(e)
};

// LPH: lanes per head = d_r / 8; kUnroll: rows in flight per lane; T1:
// tokens per workgroup.
template <int LPH, int kUnroll, int T1>
__global__ __launch_bounds__(256) void logits_kernel(LogitsArgs a) {
  constexpr int d_r = LPH * 8;
  const int b = blockIdx.y;
  const int blk = blockIdx.x;
  const int L_b = clampi(a.seq_lens[b], 0, a.L_max);
  if (blk == 0 && a.hist) {
    int32_t* h = a.hist + (size_t)b * a.n_sets * kTopkBins;
    for (int i = threadIdx.x; i < a.n_sets * kTopkBins; i += 256) h[i] = 0;
  }
  const int t_begin = blk * T1;
  if (t_begin >= L_b) return;  // uniform for the workgroup
  const int n_tok = min(T1, L_b - t_begin);

  const int cpt = a.H_r * LPH;  // 16-byte chunks per token row
  const int tpi = 256 / cpt;    // tokens per pass of the workgroup
  const int tid = threadIdx.x;
  const int slot = tid / cpt;
  const int c = tid - slot * cpt;
  const int h = c / LPH;
  const int part = c - h * LPH;

  __shared__ float lg[T1 * 17];  // [token][head], H_r <= 16; pitch 17 spreads the banks

  if (slot < tpi) {  // whole LPH lane groups are in or out together
    float qv[8];
    unpack8(ldg16(a.q_r + ((size_t)b * a.H_r + h) * d_r + part * 8), qv);
#pragma unroll
    for (int e = 0; e < 8; ++e) qv[e] *= a.qscale;
    const size_t row = (size_t)a.H_r * d_r;
    const uint16_t* base =
        a.k_r + (size_t)b * a.kr_stride_b + (size_t)t_begin * row + (size_t)h * d_r + part * 8;
    for (int i0 = slot; i0 < n_tok; i0 += tpi * kUnroll) {
      uint4 kv[kUnroll];
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        const int i = min(i0 + u * tpi, n_tok - 1);
        kv[u] = ldg16_stream(base + (size_t)i * row);
      }
#pragma unroll
      for (int u = 0; u < kUnroll; ++u) {
        float kf[8];
        unpack8(kv[u], kf);
        float acc = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc = fmaf(qv[e], kf[e], acc);
        acc = row_sum<LPH>(acc);
        const int i = i0 + u * tpi;
        if (part == 0 && i < n_tok) lg[i * 17 + h] = acc;
      }
    }
  }
  __syncthreads();

  // The block's logits leave in one coalesced burst after the stream (stores
  // spread through the stream cost far more: writes mixed into the reads).
  // They are device-scope stores, which pass through this XCD's L2 as they
  // are issued: the blocks are all resident at once and end together, and
  // dirty lines left in the L2s would all be written back at the kernel's
  // end, with nothing to overlap them.
  {
    // head-major: each head's logits of the block are one contiguous run
    for (int e = threadIdx.x; e < n_tok * a.H_r; e += 256) {
      const int h = e / n_tok;
      const int i = e - h * n_tok;
      __hip_atomic_store(&a.logits[((size_t)b * a.H_r + h) * a.L_max + t_begin + i],
                         lg[i * 17 + h], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }

  // Per-head block maximum and sum of exp2(l - max): 16 lanes per head.
  const int hh = tid >> 4;
  const int j = tid & 15;
  if (hh < a.H_r) {
    float m = -INFINITY;
    for (int i = j; i < n_tok; i += 16) m = fmaxf(m, lg[i * 17 + hh]);
    m = row_max<16>(m);
    float s = 0.f;
    for (int i = j; i < n_tok; i += 16) s += exp2f(lg[i * 17 + hh] - m);
    s = row_sum<16>(s);
    if (j == 0) {
      float* p = a.part + (((size_t)b * a.H_r + hh) * a.n_blk + blk) * 2;
      p[0] = m;
      p[1] = s;
    }
  }
}

struct SoftArgs {
  const float* logits;
  const float* part;
  const int32_t* seq_lens;
  float* scores;   // [B][n_sets][L_max]
  int32_t* hist;   // [B][n_sets][4096]: histogram of key bits 31..20 of the scores
  int L_max, H_r, n_blk, n_sets;
  int tpb;         // tokens per block of the logits kernel
};

// One workgroup per (T2 tokens, score row); thread = 4 consecutive tokens.
// A score row is a sequence (n_sets = 1: the heads' weights summed) or one
// KV head of a sequence (n_sets = H_kv: the maximum over the H_r / n_sets
// heads of its group).
// Every load is issued before the sequence length arrives (they are all
// independent of it): the thread's logits, clamped into the row, and every
// per-block pair of its head, later masked to the sequence's blocks.  One
// memory round trip precedes the arithmetic.
__global__ __launch_bounds__(256) void softmax_headsum_kernel(SoftArgs a) {
  __shared__ float c_h[16];
  __shared__ float2 wred[4];
  __shared__ int sh_hist[kTopkBins];
  const int row = blockIdx.y;
  const int b = row / a.n_sets;
  const int per = a.H_r / a.n_sets;         // heads of this row
  const int h0 = (row - b * a.n_sets) * per;  // its first head
  const bool sum_heads = a.n_sets == 1;
  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * T2;
  const int t1 = min(t0 + T2, a.L_max);
  const int L_raw = a.seq_lens[b];
  float* out = a.scores + (size_t)row * a.L_max;
  for (int i = tid; i < kTopkBins; i += 256) sh_hist[i] = 0;

  // This thread's logits (4 tokens x the row's heads, at most 16), head-major
  // rows: one float4 holds this thread's 4 tokens of a head.
  const int H_r = a.H_r;
  const int tb = t0 + 4 * tid;
  float lv[4][16];
  const bool vec = (a.L_max & 3) == 0 && tb + 3 < a.L_max;
#pragma unroll
  for (int h = 0; h < 16; ++h) {
    if (h < per) {
      const float* l = a.logits + ((size_t)b * H_r + h0 + h) * a.L_max;  // head row
      if (vec) {
        const float4 v = *reinterpret_cast<const float4*>(l + tb);
        lv[0][h] = v.x;
        lv[1][h] = v.y;
        lv[2][h] = v.z;
        lv[3][h] = v.w;
      } else {  // row tail: clamped into the row; values past the length are unused
#pragma unroll
        for (int e = 0; e < 4; ++e) lv[e][h] = l[min(tb + e, a.L_max - 1)];
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) lv[e][h] = 0.f;
    }
  }
  HeadNorm nrm;
  head_norm_load<false>(nrm, a.part, b, H_r, h0, per, a.n_blk);

  const int L_b = clampi(L_raw, 0, a.L_max);
  if (t0 >= L_b) {  // uniform: the block lies past the sequence
    for (int t = t0 + tid; t < t1; t += 256) out[t] = -INFINITY;
    return;
  }
  head_norm_finish(nrm, (L_b + a.tpb - 1) / a.tpb, c_h, wred);

#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const int t = tb + e;
    if (t >= t1) break;
    float sc = -INFINITY;
    if (t < L_b) {
      sc = 0.f;
#pragma unroll
      for (int h = 0; h < 16; ++h)
        if (h < per) {
          const float w = exp2f(lv[e][h] - c_h[h]);
          sc = sum_heads ? sc + w : fmaxf(sc, w);
        }
      atomicAdd(&sh_hist[order_key(sc) >> 20], 1);
    }
    out[t] = sc;
  }
  __syncthreads();
  int32_t* gh = a.hist + (size_t)row * kTopkBins;
  for (int i = tid; i < kTopkBins; i += 256)
    if (sh_hist[i]) atomicAdd(&gh[i], sh_hist[i]);
}

// Large grids run at most kLogitsPerCU workgroups per CU (dynamic LDS is
// reserved for the purpose): with eight per CU (what registers and LDS
// allow), 2048 workgroups of 256 tokens scored 32 sequences of 16K tokens
// ~8 us slower than with four, the grid then running in two rounds.
constexpr int kLogitsPerCU = 4;
constexpr size_t kLogitsLdsPerCU = 160 * 1024;
constexpr size_t logits_lds_reserve(int tpb) {
  // a workgroup then holds just under a quarter of the CU's LDS: four fit, five do not
  return kLogitsLdsPerCU / kLogitsPerCU - 2048 - sizeof(float) * tpb * 17;
}

template <int LPH>
void logits_dispatch(dim3 g, int tpb, bool wide, const LogitsArgs& a, hipStream_t s) {
  if (tpb == 256) {
    if (wide) logits_kernel<LPH, kUnrollWide, 256><<<g, 256, logits_lds_reserve(256), s>>>(a);
    else logits_kernel<LPH, kUnrollNarrow, 256><<<g, 256, 0, s>>>(a);
  } else if (tpb == 128) {
    logits_kernel<LPH, kUnrollNarrow, 128><<<g, 256, 0, s>>>(a);
  } else {
    logits_kernel<LPH, kUnrollNarrow, 64><<<g, 256, 0, s>>>(a);
  }
}

}  // namespace

hipError_t launch_logits(const Dims& d, const uint16_t* q_r, const uint16_t* k_r,
                         const int32_t* seq_lens, void* ws, bool zero_hist, hipStream_t s) {
  const int n_blk = score_blocks(d);
  LogitsArgs la{q_r, k_r, seq_lens, score_ws_logits(ws), score_ws_part(d, ws),
                zero_hist ? score_ws_hist(d, ws) : nullptr, d.kr_stride_b,
                d.L_max, d.H_r, n_blk, d.n_sets, d.scale_r * kLog2e};
  const int tpb = score_tokens_per_block(d);
  const dim3 g1(n_blk, d.B);
  const bool wide = (int64_t)n_blk * d.B >= 2 * (int64_t)device_cu_count();
  if (d.d_r == 64)
    logits_dispatch<8>(g1, tpb, wide, la, s);
  else
    logits_dispatch<16>(g1, tpb, wide, la, s);
  return hipGetLastError();
}

hipError_t launch_score(const Dims& d, const uint16_t* q_r, const uint16_t* k_r,
                        const int32_t* seq_lens, float* scores, void* ws,
                        hipStream_t s) {
  hipError_t e = launch_logits(d, q_r, k_r, seq_lens, ws, true, s);
  if (e != hipSuccess) return e;
  SoftArgs sa{score_ws_logits(ws), score_ws_part(d, ws), seq_lens, scores, score_ws_hist(d, ws),
              d.L_max, d.H_r, score_blocks(d), d.n_sets, score_tokens_per_block(d)};
  const dim3 g2((d.L_max + T2 - 1) / T2, d.B * d.n_sets);
  softmax_headsum_kernel<<<g2, 256, 0, s>>>(sa);
  return hipGetLastError();
}

}  // namespace spec
