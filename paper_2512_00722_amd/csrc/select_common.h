// Workgroup-wide primitives of the exact top-k selection (SpeContext Sec.
// 4.3): a two-value exclusive scan and the search for the radix bin that
// holds the k-th largest key.  Shared by the tiled selection kernels and the
// one-workgroup-per-row kernel.
#pragma once
#include "device_common.h"
#include "internal.h"

namespace spec {

// Exclusive scan of two ints over a workgroup of NT threads; returns the
// totals too.  Must be called by all threads.
template <int NT>
__device__ __forceinline__ void block_scan2(int a, int b, int& ea, int& eb, int& ta, int& tb,
                                            int* sh /* [2*NT/64] */) {
  constexpr int NW = NT / 64;
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
    sh[NW + wave] = ib;
  }
  __syncthreads();
  if (wave == 0) {
    int wa = lane < NW ? sh[lane] : 0;
    int wb = lane < NW ? sh[NW + lane] : 0;
#pragma unroll
    for (int off = 1; off < NW; off <<= 1) {
      const int na = __shfl_up(wa, off);
      const int nb = __shfl_up(wb, off);
      if (lane >= off) {
        wa += na;
        wb += nb;
      }
    }
    if (lane < NW) {
      sh[lane] = wa;  // inclusive prefix over waves
      sh[NW + lane] = wb;
    }
  }
  __syncthreads();
  const int pa = wave > 0 ? sh[wave - 1] : 0;
  const int pb = wave > 0 ? sh[NW + wave - 1] : 0;
  ea = pa + ia - a;
  eb = pb + ib - b;
  ta = sh[NW - 1];
  tb = sh[2 * NW - 1];
  __syncthreads();  // sh is reused by the next call
}

// Among `nbins` descending bins held by the workgroup (thread i owns bins
// nbins-1-i*bpt .. with bpt = max(1, nbins/NT)), find the bin where the
// running count from the top first reaches `need`.  Writes the bin and the
// count of keys in higher bins to sel[0], sel[1] and the bin's count to
// sel[2].  All threads must call; the result is valid after the call.
template <int NT>
__device__ __forceinline__ void find_bin(const int* hist, int nbins, int need, int* sh,
                                         int* sel) {
  constexpr int kMaxBpt = kTopkBins / NT;
  const int tid = threadIdx.x;
  const int bpt = nbins >= NT ? nbins / NT : 1;
  const bool owns = tid * bpt < nbins;
  int cnt[kMaxBpt];
  int local = 0;
#pragma unroll
  for (int e = 0; e < kMaxBpt; ++e) {
    cnt[e] = (owns && e < bpt) ? hist[nbins - 1 - (tid * bpt + e)] : 0;
    local += cnt[e];
  }
  int before, d0, t0, t1;
  block_scan2<NT>(local, 0, before, d0, t0, t1, sh);
  if (owns) {
#pragma unroll
    for (int e = 0; e < kMaxBpt; ++e) {
      if (e < bpt) {
        if (before < need && need <= before + cnt[e]) {
          sel[0] = nbins - 1 - (tid * bpt + e);
          sel[1] = before;
          sel[2] = cnt[e];
        }
        before += cnt[e];
      }
    }
  }
  __syncthreads();
}

}  // namespace spec
