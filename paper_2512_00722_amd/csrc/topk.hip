// Exact top-k token selection on gfx950 (SpeContext Sec. 4.3: the important
// tokens are chosen from the retrieval head's attention weights).
//
// Scores are mapped to order-preserving 32-bit keys.  The k-th largest key T
// is located from the top 12 key bits first: a 4096-bin histogram of every
// sequence (built while the scores are written, or by topk_hist_kernel for a
// standalone call) names the bin b1 holding the k-th key, the number c1 of
// keys in higher bins (all selected) and the bin's population n1.
//
// Two kernels follow the histogram:
//  * topk_classify_kernel, one 256-thread workgroup per 2048-token tile,
//    recomputes b1 from the histogram (tile 0 also hands b1, c1, n1 on) and
//    appends, in token order, the tile's tokens of higher bins and its
//    bin-b1 candidates (key, token) to per-tile lists (wave-ordered appends
//    with ballots, coalesced loads);
//  * topk_select_kernel, one 1024-thread workgroup per sequence, loads b1
//    with the per-tile counts, gathers the lists into LDS by prefix sums,
//    resolves the remaining 20 key bits of T among the candidates only (two
//    10-bit LDS histogram passes), which also gives r, the number of keys
//    equal to T to take (the lowest-index ones), compacts the selected
//    candidates in order and merges the two ascending lists by binary
//    search.
//  * When the lists would not fit (more than 8192 tokens above the bin or
//    12288 candidates) the select kernel falls back to a general path: two
//    more radix passes over the row (bits 19..8, 7..0) and an ordered
//    compaction with one workgroup scan per 4096 tokens.
// Both paths write the indices ascending, so no sort is needed.
#include "device_common.h"
#include "internal.h"
#include "select_common.h"

namespace spec {
namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / 64;
constexpr int kBins = kTopkBins;  // 4096: key bits 31..20
constexpr int kGtCap = 8192;
constexpr int kCandCap = 12288;
constexpr int kTile = kTopkTile;  // tokens per classify workgroup
constexpr int kMaxTiles = 1024;   // fast path: at most one tile per select thread

// Key of row[t] for t < L, else 0 (below every real key).  The load is
// unconditional, from an index clamped into [0, row_len): a conditional load
// makes the compiler wait for each one before the next is issued.
__device__ __forceinline__ uint32_t key_at(const float* row, int t, int L, int row_len) {
  const float v = row[min(max(t, 0), row_len - 1)];
  // a mask, not a select: a select lets the compiler sink the load into a branch
  const uint32_t keep = 0u - (uint32_t)(t < L);
  return order_key(v) & keep;
}

// Copy a [kBins] int array from global memory to LDS with NT threads: all
// loads of a thread are issued before the first LDS write.
template <int NT>
__device__ __forceinline__ void load_hist(const int32_t* g, int* sh) {
  constexpr int kPer = kBins / NT;
  int v[kPer];
#pragma unroll
  for (int e = 0; e < kPer; ++e) v[e] = g[threadIdx.x + e * NT];
#pragma unroll
  for (int e = 0; e < kPer; ++e) sh[threadIdx.x + e * NT] = v[e];
}

// Per-tile lists written by the classify kernel (workspace).
struct TileLists {
  int32_t* sel;     // [B][4]: b1, c1, n1 of the histogram (classify's tile 0 writes them)
  int32_t* cnt;     // [B][n_tiles][2]: tokens above bin b1, candidates in b1
  int32_t* gt;      // [B][n_tiles][kTile]
  uint32_t* ckey;   // [B][n_tiles][kTile]
  int32_t* cidx;    // [B][n_tiles][kTile]
  int n_tiles;      // ceil(L_max / kTile)
};

struct SelArgs {
  const float* scores;  // [B][L_max]
  const int32_t* seq_lens;
  const int32_t* ks;
  int32_t* idx;         // [B][k_max]
  int32_t* counts;      // [B] or null
  TileLists tl;
  int L_max, k_max, n_sets;  // score rows: B * n_sets, sequence = row / n_sets
};

// Merge of two ascending lists of distinct values, a (n entries) and b (m),
// into out[0 .. n+m): thread t writes outputs [t q, t q + q), q = ceil((n+m)
// / threads).  Its starting split (i from a, d - i from b) is found by one
// binary search along the diagonal d = t q; the q outputs follow in order.
__device__ __forceinline__ void merge_path(const int* a, int n, const int* b, int m,
                                           int32_t* out) {
  const int total = n + m;
  const int q = (total + kThreads - 1) / kThreads;
  int d = threadIdx.x * q;
  if (d >= total) return;
  int lo = max(0, d - m), hi = min(d, n);
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (a[mid] < b[d - 1 - mid]) lo = mid + 1; else hi = mid;
  }
  int i = lo, j = d - lo;
  const int end = min(d + q, total);
  for (; d < end; ++d) {
    if (j >= m || (i < n && a[i] < b[j])) out[d] = a[i++];
    else out[d] = b[j++];
  }
}

__global__ __launch_bounds__(kThreads) void topk_select_kernel(SelArgs a) {
  __shared__ int s_hist[kBins];
  __shared__ int s_gt[kGtCap];
  __shared__ uint32_t s_ckey[kCandCap];
  __shared__ int s_cidx[kCandCap];
  __shared__ int s_scan[2 * kWaves];
  __shared__ int s_sel[4];

  const int srow = blockIdx.x;      // score row
  const int b = srow / a.n_sets;    // its sequence
  const int tid = threadIdx.x;
  const int L_b = clampi(a.seq_lens[b], 0, a.L_max);
  const int k_b = clampi(a.ks[b], 0, min(L_b, a.k_max));
  const float* row = a.scores + (size_t)srow * a.L_max;
  int32_t* out = a.idx + (size_t)srow * a.k_max;

  if (tid == 0) s_sel[0] = s_sel[1] = s_sel[2] = -1;
  if (tid == 0 && a.counts && srow == b * a.n_sets) a.counts[b] = k_b;
  for (int j = k_b + tid; j < a.k_max; j += kThreads) out[j] = -1;
  if (k_b == 0 || k_b == L_b) {  // nothing, or every token, is selected
    for (int j = tid; j < k_b; j += kThreads) out[j] = j;
    return;
  }

  // ---- the bin b1 of the k-th key (the classify kernel found it in the
  // 12-bit histogram), loaded with the per-tile list counts: one round trip
  const int n_tiles_b = (L_b + kTile - 1) / kTile;
  const int32_t* tcnt = a.tl.cnt + (size_t)srow * a.tl.n_tiles * 2;
  const int tcl = min(tid, a.tl.n_tiles - 1);  // clamped: the load is unconditional
  int tg = tcnt[2 * tcl];
  int tc = tcnt[2 * tcl + 1];
  if (!(tid < n_tiles_b && n_tiles_b <= kMaxTiles)) tg = tc = 0;
  const int b1i = a.tl.sel[srow * 4];
  const int c1 = a.tl.sel[srow * 4 + 1];  // keys in higher bins: all selected
  const int n1 = a.tl.sel[srow * 4 + 2];  // keys in bin b1
  const int r1 = k_b - c1;                // keys still to take from bin b1 (1 <= r1 <= n1)
  const uint32_t b1 = (uint32_t)b1i;
  // A histogram that does not describe this row (never produced by this
  // library) sends the sequence down the general path from scratch.
  const bool hist_ok = b1i >= 0 && b1i < kBins && c1 >= 0 && c1 < k_b && r1 <= n1;

  if (hist_ok && c1 <= kGtCap && n1 <= kCandCap && n_tiles_b <= kMaxTiles) {
    // ---------------- fast path: gather the per-tile lists ----------------
    // Per-tile offsets and counts go to the histogram's LDS (no longer
    // needed); then each wave copies whole tiles, four at a time, with
    // coalesced, unconditional loads.
    int* s_off_g = s_hist;
    int* s_off_c = s_hist + kMaxTiles;
    int* s_cnt_g = s_hist + 2 * kMaxTiles;
    int* s_cnt_c = s_hist + 3 * kMaxTiles;
    if (n_tiles_b <= 64) {  // up to 128K tokens: one wavefront scans the counts
      if (tid < 64) {
        int ig = tg, ic = tc;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
          const int ng = __shfl_up(ig, off);
          const int nc = __shfl_up(ic, off);
          if (tid >= off) {
            ig += ng;
            ic += nc;
          }
        }
        if (tid < n_tiles_b) {
          s_off_g[tid] = ig - tg;
          s_off_c[tid] = ic - tc;
          s_cnt_g[tid] = tg;
          s_cnt_c[tid] = tc;
        }
      }
    } else {
      int og, oc, sum_g, sum_c;
      block_scan2<kThreads>(tg, tc, og, oc, sum_g, sum_c, s_scan);
      if (tid < n_tiles_b) {
        s_off_g[tid] = og;
        s_off_c[tid] = oc;
        s_cnt_g[tid] = tg;
        s_cnt_c[tid] = tc;
      }
    }
    __syncthreads();
    const int lane = tid & 63;
    const int wv = tid >> 6;
    const int32_t* tgt = a.tl.gt + (size_t)srow * a.tl.n_tiles * kTile;
    const uint32_t* tck = a.tl.ckey + (size_t)srow * a.tl.n_tiles * kTile;
    const int32_t* tci = a.tl.cidx + (size_t)srow * a.tl.n_tiles * kTile;
    auto put = [&](int t, int i, int gv, uint32_t kv, int iv) {
      if (i < s_cnt_g[t] && s_off_g[t] + i < kGtCap) s_gt[s_off_g[t] + i] = gv;
      if (i < s_cnt_c[t] && s_off_c[t] + i < kCandCap) {
        s_ckey[s_off_c[t] + i] = kv;
        s_cidx[s_off_c[t] + i] = iv;
      }
    };
    for (int t0 = wv; t0 < n_tiles_b; t0 += 4 * kWaves) {
      int gv[4], iv[4];
      uint32_t kv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const size_t q = (size_t)min(t0 + u * kWaves, n_tiles_b - 1) * kTile + lane;
        gv[u] = tgt[q];
        kv[u] = tck[q];
        iv[u] = tci[q];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int t = t0 + u * kWaves;
        if (t < n_tiles_b) {
          put(t, lane, gv[u], kv[u], iv[u]);
          // tiles with more than 64 entries in a list (the heavy tokens
          // crowd a few tiles): four rounds of loads in flight at a time
          const int n = max(s_cnt_g[t], s_cnt_c[t]);
          for (int i0 = 64; i0 < n; i0 += 256) {
            int gr[4], ir[4];
            uint32_t kr[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const size_t q = (size_t)t * kTile + min(i0 + 64 * r + lane, kTile - 1);
              gr[r] = tgt[q];
              kr[r] = tck[q];
              ir[r] = tci[q];
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) put(t, i0 + 64 * r + lane, gr[r], kr[r], ir[r]);
          }
        }
      }
    }
    __syncthreads();

    // ---- resolve the low 20 bits of T among the n1 candidates
    int remaining = r1;
    uint32_t T = b1 << 20;
#pragma unroll 1
    for (int pass = 0; pass < 2; ++pass) {
      const int shift = pass == 0 ? 10 : 0;
      for (int i = tid; i < 1024; i += kThreads) s_hist[i] = 0;
      __syncthreads();
      const uint32_t hi_mask = pass == 0 ? 0xFFF00000u : 0xFFFFFC00u;
      for (int i = tid; i < n1; i += kThreads) {
        const uint32_t kk = s_ckey[i];
        if ((kk & hi_mask) == T) atomicAdd(&s_hist[(kk >> shift) & 1023], 1);
      }
      __syncthreads();
      find_bin<kThreads>(s_hist, 1024, remaining, s_scan, s_sel);
      T |= (uint32_t)s_sel[0] << shift;
      remaining -= s_sel[1];
      __syncthreads();
    }
    const int r = remaining;  // keys equal to T to take, lowest index first

    // ---- selected candidates, in token order, into s_ckey (as ints)
    const int cseg = (n1 + kThreads - 1) / kThreads;  // <= 12
    const int c0 = min(tid * cseg, n1);
    const int cend = min(c0 + cseg, n1);
    uint32_t ck[12];
    int ci[12];
    int ngtT = 0, neqT = 0;
#pragma unroll
    for (int e = 0; e < 12; ++e) {
      const bool v = c0 + e < cend;
      ck[e] = v ? s_ckey[c0 + e] : 0u;
      ci[e] = v ? s_cidx[c0 + e] : 0;
      ngtT += v && ck[e] > T;
      neqT += v && ck[e] == T;
    }
    int gbef, ebef, gtot, etot;
    block_scan2<kThreads>(ngtT, neqT, gbef, ebef, gtot, etot, s_scan);  // also orders the reads above
    int* s_selv = reinterpret_cast<int*>(s_ckey);
#pragma unroll
    for (int e = 0; e < 12; ++e) {
      if (c0 + e < cend) {
        if (ck[e] > T) {
          s_selv[gbef + min(ebef, r)] = ci[e];
          ++gbef;
        } else if (ck[e] == T) {
          if (ebef < r) s_selv[gbef + ebef] = ci[e];
          ++ebef;
        }
      }
    }
    __syncthreads();

    // ---- merge the two ascending lists (c1 + r1 = k_b entries)
    merge_path(s_gt, c1, s_selv, r1, out);
    return;
  }

  // ---------------- general path: radix passes over the row ----------------
  uint32_t prefix = hist_ok ? b1 << 20 : 0u;
  uint32_t mask = hist_ok ? 0xFFF00000u : 0u;
  int remaining = hist_ok ? r1 : k_b;
#pragma unroll 1
  for (int pass = hist_ok ? 1 : 0; pass < 3; ++pass) {
    const int shift = pass == 0 ? 20 : (pass == 1 ? 8 : 0);
    const int nbins = pass < 2 ? 4096 : 256;
    for (int i = tid; i < nbins; i += kThreads) s_hist[i] = 0;
    __syncthreads();
    for (int t0 = 0; t0 < L_b; t0 += 8 * kThreads) {
      uint32_t k8[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) k8[e] = key_at(row, t0 + e * kThreads + tid, L_b, a.L_max);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (t0 + e * kThreads + tid < L_b && (k8[e] & mask) == prefix)
          atomicAdd(&s_hist[(k8[e] >> shift) & (nbins - 1)], 1);
    }
    __syncthreads();
    find_bin<kThreads>(s_hist, nbins, remaining, s_scan, s_sel);
    prefix |= (uint32_t)s_sel[0] << shift;
    mask |= (uint32_t)(nbins - 1) << shift;
    remaining -= s_sel[1];
    __syncthreads();
  }
  const uint32_t T = prefix;
  const int r = remaining;

  int carry_gt = 0, carry_eq = 0;
  for (int base = 0; base < L_b; base += 4 * kThreads) {
    const int t0 = base + 4 * tid;
    uint32_t key[4];
    int ngt = 0, neq = 0;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      key[e] = key_at(row, t0 + e, L_b, a.L_max);
      const bool valid = t0 + e < L_b;
      ngt += (valid && key[e] > T);
      neq += (valid && key[e] == T);
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

constexpr int kClsThreads = 256;
constexpr int kClsWaves = kClsThreads / 64;
constexpr int kClsPerLane = kTile / kClsThreads;  // 8 tokens per lane

struct ClsArgs {
  const float* scores;
  const int32_t* seq_lens;
  const int32_t* ks;
  const int32_t* hist;
  TileLists tl;
  int L_max, k_max, n_sets;  // score rows: B * n_sets, sequence = row / n_sets
};

// grid (n_tiles, B).  Wave w of a tile owns tokens [t0 + 512w, t0 + 512w + 512);
// lane i reads tokens base + 64j + i.  An element's list slot is its wave's
// offset plus the flagged elements before it in (j, lane) order.
__global__ __launch_bounds__(kClsThreads) void topk_classify_kernel(ClsArgs a) {
  __shared__ int s_hist[kBins];
  __shared__ int s_scan[2 * kClsWaves];
  __shared__ int s_sel[4];
  __shared__ int s_wcnt[2 * kClsWaves];
  const int srow = blockIdx.y;  // score row
  const int b = srow / a.n_sets;
  const int tile = blockIdx.x;
  const int tid = threadIdx.x;
  const int t0 = tile * kTile;

  // The lengths, the tile's scores and the histogram are independent: all
  // are requested before any is used (the scores clamped into the row, and
  // masked to the sequence once its length has arrived).
  const int L_raw = a.seq_lens[b];
  const int k_raw = a.ks[b];
  const float* row = a.scores + (size_t)srow * a.L_max;
  const int lane = tid & 63;
  const int wv = tid >> 6;
  const int w0 = t0 + wv * (kTile / kClsWaves);
  float sv[kClsPerLane];
#pragma unroll
  for (int j = 0; j < kClsPerLane; ++j) sv[j] = row[min(w0 + 64 * j + lane, a.L_max - 1)];
  load_hist<kClsThreads>(a.hist + (size_t)srow * kBins, s_hist);
  const int L_b = clampi(L_raw, 0, a.L_max);
  const int k_b = clampi(k_raw, 0, min(L_b, a.k_max));
  if (k_b == 0 || k_b == L_b || t0 >= L_b) return;  // uniform: nothing to classify
  const int w1 = min(w0 + kTile / kClsWaves, L_b);
  uint32_t kk[kClsPerLane];
#pragma unroll
  for (int j = 0; j < kClsPerLane; ++j)  // a mask, not a select (see key_at)
    kk[j] = order_key(sv[j]) & (0u - (uint32_t)(w0 + 64 * j + lane < w1));
  if (tid == 0) s_sel[0] = s_sel[1] = s_sel[2] = -1;
  __syncthreads();
  find_bin<kClsThreads>(s_hist, kBins, k_b, s_scan, s_sel);
  const int b1i = s_sel[0], c1 = s_sel[1], n1 = s_sel[2];
  if (tile == 0 && tid == 0) {  // for the select kernel, valid or not
    a.tl.sel[srow * 4] = b1i;
    a.tl.sel[srow * 4 + 1] = c1;
    a.tl.sel[srow * 4 + 2] = n1;
  }
  // Same decision as the select kernel: it only reads the lists on its fast path.
  if (!(b1i >= 0 && c1 >= 0 && c1 < k_b && k_b - c1 <= n1) || c1 > kGtCap || n1 > kCandCap)
    return;
  const uint32_t b1 = (uint32_t)b1i;
  int wgt = 0, wcand = 0;
#pragma unroll
  for (int j = 0; j < kClsPerLane; ++j) {
    const bool in = w0 + 64 * j + lane < w1;
    const uint32_t dg = kk[j] >> 20;
    wgt += __popcll(__ballot(in && dg > b1));
    wcand += __popcll(__ballot(in && dg == b1));
  }
  if (lane == 0) {
    s_wcnt[wv] = wgt;
    s_wcnt[kClsWaves + wv] = wcand;
  }
  __syncthreads();
  int gpos = 0, cpos = 0, gtot = 0, ctot = 0;
#pragma unroll
  for (int i = 0; i < kClsWaves; ++i) {
    if (i < wv) {
      gpos += s_wcnt[i];
      cpos += s_wcnt[kClsWaves + i];
    }
    gtot += s_wcnt[i];
    ctot += s_wcnt[kClsWaves + i];
  }
  const size_t tb = ((size_t)srow * a.tl.n_tiles + tile);
  int32_t* gt = a.tl.gt + tb * kTile;
  uint32_t* ck = a.tl.ckey + tb * kTile;
  int32_t* ci = a.tl.cidx + tb * kTile;
  const uint64_t lt_mask = (1ull << lane) - 1ull;
#pragma unroll
  for (int j = 0; j < kClsPerLane; ++j) {
    const int t = w0 + 64 * j + lane;
    const bool in = t < w1;
    const uint32_t dg = kk[j] >> 20;
    const uint64_t mg = __ballot(in && dg > b1);
    const uint64_t mc = __ballot(in && dg == b1);
    if (in && dg > b1) {
      gt[gpos + __popcll(mg & lt_mask)] = t;
    } else if (in && dg == b1) {
      const int q = cpos + __popcll(mc & lt_mask);
      ck[q] = kk[j];
      ci[q] = t;
    }
    gpos += __popcll(mg);
    cpos += __popcll(mc);
  }
  if (tid == 0) {
    a.tl.cnt[tb * 2] = gtot;
    a.tl.cnt[tb * 2 + 1] = ctot;
  }
}

// Standalone histogram of key bits 31..20 (the score kernels build the same
// histogram on the fly).  grid (ceil(L_max / 4096), B); hist pre-zeroed.
__global__ __launch_bounds__(256) void topk_hist_kernel(const float* scores,
                                                        const int32_t* seq_lens,
                                                        int32_t* hist, int L_max, int n_sets) {
  __shared__ int sh[kBins];
  const int srow = blockIdx.y;  // score row; its sequence is srow / n_sets
  const int L_b = clampi(seq_lens[srow / n_sets], 0, L_max);
  const int t0 = blockIdx.x * 4096;
  if (t0 >= L_b) return;
  for (int i = threadIdx.x; i < kBins; i += 256) sh[i] = 0;
  __syncthreads();
  const float* row = scores + (size_t)srow * L_max;
  const int t1 = min(t0 + 4096, L_b);
  float v[16];  // 4096 / 256 tokens per thread, all loads in flight
#pragma unroll
  for (int e = 0; e < 16; ++e) v[e] = row[min(t0 + (int)threadIdx.x + 256 * e, t1 - 1)];
#pragma unroll
  for (int e = 0; e < 16; ++e)
    if (t0 + (int)threadIdx.x + 256 * e < t1) atomicAdd(&sh[order_key(v[e]) >> 20], 1);
  __syncthreads();
  int32_t* gh = hist + (size_t)srow * kBins;
  for (int i = threadIdx.x; i < kBins; i += 256)
    if (sh[i]) atomicAdd(&gh[i], sh[i]);
}

__global__ __launch_bounds__(256) void zero_kernel(int32_t* p, int n) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0;
}

TileLists tile_lists(const Dims& d, void* lists) {
  TileLists tl;
  const int n_tiles = topk_tiles(d);
  const size_t n = (size_t)d.B * d.n_sets * n_tiles;
  char* p = static_cast<char*>(lists);
  tl.sel = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * 4 * (size_t)d.B * d.n_sets);
  tl.cnt = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * 2 * n);
  tl.gt = reinterpret_cast<int32_t*>(p);
  p += align_up(sizeof(int32_t) * n * kTile);
  tl.ckey = reinterpret_cast<uint32_t*>(p);
  p += align_up(sizeof(uint32_t) * n * kTile);
  tl.cidx = reinterpret_cast<int32_t*>(p);
  tl.n_tiles = n_tiles;
  return tl;
}

}  // namespace

hipError_t launch_topk_select(const Dims& d, const float* scores, const int32_t* seq_lens,
                              const int32_t* ks, const int32_t* hist, void* lists, int32_t* idx,
                              int32_t* counts, hipStream_t s) {
  const TileLists tl = tile_lists(d, lists);
  ClsArgs c{scores, seq_lens, ks, hist, tl, d.L_max, d.k_max, d.n_sets};
  topk_classify_kernel<<<dim3(tl.n_tiles, d.B * d.n_sets), kClsThreads, 0, s>>>(c);
  SelArgs a{scores, seq_lens, ks, idx, counts, tl, d.L_max, d.k_max, d.n_sets};
  topk_select_kernel<<<d.B * d.n_sets, kThreads, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_topk(const Dims& d, const float* scores, const int32_t* seq_lens,
                       const int32_t* ks, int32_t* idx, int32_t* counts, void* ws,
                       hipStream_t s) {
  if (row_select_fits(d, 1))  // short rows: one workgroup per row, keys in LDS
    return launch_row_select(d, nullptr, const_cast<float*>(scores), seq_lens, ks, idx, counts,
                             s);
  int32_t* hist = static_cast<int32_t*>(ws);
  const int n = d.B * d.n_sets * kBins;
  zero_kernel<<<(n + 255) / 256, 256, 0, s>>>(hist, n);
  const dim3 g((d.L_max + 4095) / 4096, d.B * d.n_sets);
  topk_hist_kernel<<<g, 256, 0, s>>>(scores, seq_lens, hist, d.L_max, d.n_sets);
  return launch_topk_select(d, scores, seq_lens, ks, hist,
                            static_cast<char*>(ws) + topk_hist_bytes(d), idx, counts, s);
}

}  // namespace spec
