// Per-head softmax normalisers of one score row (SpeContext Sec. 4.3, Eq. 1:
// the softmax over a sequence's tokens, per retrieval head).  The logits
// kernel leaves, per block of tokens and head, the pair (block max, sum of
// exp2(l - max)); the normaliser of head h is c_h = M_h + log2 Z_h over the
// blocks that hold the sequence.  Shared by the softmax/head-sum kernel and
// the one-workgroup-per-row selection kernel, so that both form the same
// scores bit for bit.
#pragma once
#include "device_common.h"

namespace spec {

// The first 256 threads of the workgroup merge: 256/P lanes per head (P the
// row's head count rounded up to a power of two), 16 pairs in flight per
// lane, then a butterfly over the head's lanes of the wave and, for heads
// wider than a wave, a combine of the per-wave results.
struct HeadNorm {
  float2 pv[16];
  const float2* pp;  // the head's pairs (head-major: contiguous)
  int per, lph, hh, j;
};

// Issues the pair loads; they depend on nothing but the row.  Pairs of
// blocks past the sequence (not written by this call) are loaded with the
// rest, clamped into the row, and masked by head_norm_finish.  kWide: the
// workgroup has more than 256 threads (the others load nothing).
template <bool kWide>
__device__ __forceinline__ void head_norm_load(HeadNorm& n, const float* part, int b, int H_r,
                                               int h0, int per, int n_blk) {
  const int P = per <= 1 ? 1 : per <= 2 ? 2 : per <= 4 ? 4 : per <= 8 ? 8 : 16;
  n.per = per;
  n.lph = 256 / P;
  n.hh = (int)threadIdx.x / n.lph;
  n.j = (int)threadIdx.x - n.hh * n.lph;
  n.pp = reinterpret_cast<const float2*>(part) +
         ((size_t)b * H_r + h0 + min(n.hh, per - 1)) * n_blk;
  if (kWide && threadIdx.x >= 256) {
#pragma unroll
    for (int u = 0; u < 16; ++u) n.pv[u] = make_float2(-INFINITY, 0.f);
    return;
  }
#pragma unroll
  for (int u = 0; u < 16; ++u) n.pv[u] = n.pp[min(n.j + n.lph * u, n_blk - 1)];
}

// Merges the pairs of the sequence's nb blocks into c_h[0 .. per) (LDS).
// wred: 4 float2 of LDS.  Every thread of the workgroup must call; the
// normalisers are visible to all threads on return.
__device__ __forceinline__ void head_norm_finish(const HeadNorm& n, int nb, float* c_h,
                                                 float2* wred) {
  const int tid = threadIdx.x;
  float m = -INFINITY, s = 0.f;
  if (n.hh < n.per) {  // threads past the first 256 have hh >= P >= per
#pragma unroll
    for (int u = 0; u < 16; ++u)
      if (n.j + n.lph * u < nb) ms_combine(m, s, n.pv[u].x, n.pv[u].y);
    for (int i0 = n.j + n.lph * 16; i0 < nb; i0 += n.lph * 16) {  // long rows
      float2 v[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int i = i0 + n.lph * u;
        v[u] = i < nb ? n.pp[i] : make_float2(-INFINITY, 0.f);
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) ms_combine(m, s, v[u].x, v[u].y);
    }
  }
  const int width = n.lph < 64 ? n.lph : 64;
  for (int off = 1; off < width; off <<= 1) {
    const float m2 = __shfl_xor(m, off);
    const float s2 = __shfl_xor(s, off);
    ms_combine(m, s, m2, s2);
  }
  if (n.lph <= 64) {
    if (n.j == 0 && n.hh < n.per) c_h[n.hh] = m + log2f(s);
  } else {
    if ((tid & 63) == 0 && tid < 256) wred[tid >> 6] = make_float2(m, s);
    __syncthreads();
    if (tid < n.per) {
      const int wpw = n.lph / 64;  // waves per head
      float mm = -INFINITY, ss = 0.f;
      for (int w = tid * wpw; w < (tid + 1) * wpw; ++w) ms_combine(mm, ss, wred[w].x, wred[w].y);
      c_h[tid] = mm + log2f(ss);
    }
  }
  __syncthreads();
}

}  // namespace spec
