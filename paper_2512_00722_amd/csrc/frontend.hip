// Retrieval-head front end for the new token of every sequence (Sec. 4.3:
// the retrieval head keeps only the embedding and the Q/K projection of the
// distilled model, whose 2K training context is extended with YaRN):
//
//   x      = emb[token_b]                                   [hidden]
//   q, k   = W_q x, W_k x                                   [H_r][d_r] each
//   q_r[b] = m * R(pos_b) q,   K_r[b, pos_b] = m * R(pos_b) k
//
// R(pos) turns dimension pair (i, i + d_r/2) of every head by pos * theta'_i,
// theta'_i being the rotary frequency after YaRN interpolation and m YaRN's
// magnitude factor.
//
// The projections are one skinny GEMM, [B x hidden] . [hidden x 2*H_r*d_r],
// whose weights (2 * H_r * d_r * hidden bf16, 8-32 MiB) are read once per call
// for the whole batch: the work is bound by HBM bandwidth on them, and one
// CU streams only about 30 GB/s, so every CU must take part.
//
// Up to 16 sequences: one kernel, qk_gemv_kernel.  A workgroup owns two
// rotary pairs (four features) of one head of Q or K over the whole hidden
// dimension (2 * H_r * d_r / 4 workgroups: 256 for 8 heads of 64).  Its
// waves take 512-element slabs of the hidden dimension in turn; per slab a
// load instruction reads 1 KiB of one weight or embedding row, and each lane
// forms fp32 dot products over its 8 elements (vector ALU: with at most 16
// tokens the matrix cores would idle on padding; v_dot2_f32_bf16 takes the
// bf16 pairs as loaded).  Lane sums are reduced
// within 16-lane rows by DPP, then over rows and waves in LDS; the pairs are
// rotated in the workgroup.  Every weight byte is read once; the embedding
// rows come from L2.
//
// More than 64 sequences: two kernels, since a narrow tile per workgroup
// would make every workgroup re-read all embedding rows.
//
//  1. qk_partial_kernel (matrix cores, v_mfma_f32_16x16x32_bf16, tokens on
//     the M side): a workgroup owns 16 output features of Q or K -- the
//     dimensions i0..i0+7 of one head and their rotary partners i0+d_r/2.. --
//     over one of KS slices of the hidden dimension (KS chosen so that the
//     grid has about two workgroups per CU).  Its 4 waves take the slice's
//     128-element steps in turn; per step a lane loads 16 bytes from each of
//     four 32-element k-slices of its weight row (feature) and embedding row
//     (token), so that the four lanes of a row read 64 contiguous bytes per
//     load instruction; all loads of a chunk of steps are issued before the
//     first MFMA.  The waves' tiles are summed in LDS and the fp32 partial
//     tile is written to the workspace, [KS][B][2*H_r*d_r].
//     One workgroup also computes the YaRN frequencies and m (fp64) into the
//     workspace while its loads are in flight.
//  2. qk_finish_kernel: one thread per (sequence, Q/K, head, pair) sums the
//     KS partials of both pair members in slice order (deterministic), forms
//     the angle pos * theta'_i in fp64 (positions reach 2^17 and beyond) and
//     reduces it modulo 2 pi in fp64 with a two-term 2 pi, takes sin and cos
//     of the reduced angle, rotates, scales, rounds to bf16 and stores q_r or
//     the new K_r row.
#include <math.h>

#include "device_common.h"
#include "internal.h"

namespace spec {
namespace {

constexpr int kFeWaves = 4;
constexpr int kFeThreads = 64 * kFeWaves;
constexpr int kFeStep = 128;     // hidden elements per wave step: 4 k-slices of 32
constexpr int kFeBlocksTarget = 512;
constexpr int kFinishThreads = 256;

struct FrontArgs {
  const int32_t* tokens;
  const int32_t* pos;
  const uint16_t* emb;
  const uint16_t* w_q;
  const uint16_t* w_k;
  uint16_t* q_r;
  uint16_t* k_r;
  float* part;     // [KS][B][2 * H_r * d_r]
  double* theta;   // [d_r / 2] YaRN frequencies, then the magnitude factor m
  int64_t kr_stride_b;
  int B, vocab, hidden, H_r, d_r, L_cap;
  int ks, steps_per_split;
  float base, scale, alpha, beta;
  int orig_ctx;
};

// fp32 -> bf16 bits, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint16_t to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Rotary frequency of dimension pair i after YaRN interpolation (fp64).  The
// pair turns r = orig_ctx * theta / (2 pi) times over the original context;
// the ramp gamma(r), 0 at alpha and 1 at beta, blends the frequency divided
// by the scale (gamma = 0) with the unchanged one (gamma = 1).
__device__ double yarn_theta(const FrontArgs& a, int i) {
  const double theta = pow((double)a.base, -2.0 * (double)i / (double)a.d_r);
  if (!(a.scale > 1.0f)) return theta;
  const double turns = (double)a.orig_ctx * theta / (2.0 * M_PI);
  double gamma = (turns - (double)a.alpha) / ((double)a.beta - (double)a.alpha);
  gamma = gamma < 0.0 ? 0.0 : (gamma > 1.0 ? 1.0 : gamma);
  return (1.0 - gamma) * theta / (double)a.scale + gamma * theta;
}

// Rotate one pair, scale, round and store (q_r, or the new K_r row).
__device__ __forceinline__ void store_pair(const FrontArgs& a, int mat, int b, int h, int i,
                                           float x, float y, double theta, float m) {
  const int pos = a.pos[b];
  // angle in fp64, reduced modulo 2 pi (hi + lo parts of 2 pi; |k| < 2^29
  // leaves the reduced angle accurate to about 1e-15)
  const double ang = (double)pos * theta;
  const double k = rint(ang * 0.15915494309189535);
  double red = fma(-k, 6.283185307179586, ang);
  red = fma(-k, 2.4492935982947064e-16, red);
  float sn, cs;
  sincosf((float)red, &sn, &cs);
  const float c = m * cs, s = m * sn;
  uint16_t* dst;
  if (mat == 0) {
    dst = a.q_r + ((size_t)b * a.H_r + h) * a.d_r;
  } else {
    if (pos < 0 || pos >= a.L_cap) return;  // nothing appended outside the cache
    dst = a.k_r + (size_t)b * a.kr_stride_b + ((size_t)pos * a.H_r + h) * a.d_r;
  }
  dst[i] = to_bf16(x * c - y * s);
  dst[i + a.d_r / 2] = to_bf16(x * s + y * c);
}

// T: 16-token row tiles per workgroup.  CH: wave steps whose loads are
// issued together.
template <int T, int CH>
__global__ __launch_bounds__(kFeThreads) void qk_partial_kernel(FrontArgs a) {
  __shared__ float red[kFeWaves * T * 256];

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int n_tiles = 2 * a.H_r * (a.d_r / 16);
  const int tile = blockIdx.x % n_tiles;
  const int split = blockIdx.x / n_tiles;
  const int tiles_per_head = a.d_r / 16;
  const int per_mat = a.H_r * tiles_per_head;
  const int mat = tile / per_mat;  // 0: Q, 1: K
  const int rem = tile - mat * per_mat;
  const int h = rem / tiles_per_head;
  const int i0 = 8 * (rem - h * tiles_per_head);
  const int b0 = blockIdx.y * 16 * T;
  const int n_steps = a.hidden / kFeStep;
  const int s_begin = split * a.steps_per_split;
  const int s_end = min(n_steps, s_begin + a.steps_per_split);

  // MFMA operands: lane (n, g) = (lane & 15, lane >> 4) feeds column n of B
  // (a feature) and row n of A (a token) with elements 8g..8g+7 of each
  // 32-element k-slice.
  const int n = lane & 15;
  const int g = lane >> 4;
  const int fbase = h * a.d_r + i0 + (n & 7) + (n >> 3) * (a.d_r / 2);
  const uint16_t* wrow = (mat ? a.w_k : a.w_q) + (size_t)fbase * a.hidden + 8 * g;
  const uint16_t* erow[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int b = min(b0 + 16 * t + n, a.B - 1);  // rows past B compute a copy, never stored
    const int tok = clampi(a.tokens[b], 0, a.vocab - 1);
    erow[t] = a.emb + (size_t)tok * a.hidden + 8 * g;
  }

  floatx4 acc[T];
#pragma unroll
  for (int t = 0; t < T; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};

  for (int s0 = s_begin + wave; s0 < s_end; s0 += kFeWaves * CH) {
    // Loads of the chunk, all unconditional (steps past the slice re-read
    // its last step, inside the row), issued before the first MFMA.
    uint4 w[CH][4];
    uint4 e[CH][T][4];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const size_t off = (size_t)min(s0 + c * kFeWaves, s_end - 1) * kFeStep;
#pragma unroll
      for (int j = 0; j < 4; ++j) w[c][j] = ldg16(wrow + off + 32 * j);
#pragma unroll
      for (int t = 0; t < T; ++t)
#pragma unroll
        for (int j = 0; j < 4; ++j) e[c][t][j] = ldg16(erow[t] + off + 32 * j);
    }
    __builtin_amdgcn_sched_barrier(0);  // no MFMA (and its wait) moves above a load
    if (blockIdx.x == 0 && blockIdx.y == 0 && s0 == s_begin + wave && wave == 0) {
      if (lane < a.d_r / 2) a.theta[lane] = yarn_theta(a, lane);
      if (lane == 0) a.theta[a.d_r / 2] = a.scale > 1.0f ? 0.1 * log((double)a.scale) + 1.0 : 1.0;
    }
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      if (s0 + c * kFeWaves < s_end) {  // wave-uniform
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, e[c][t][j]), __builtin_bit_cast(bf16x8, w[c][j]),
                acc[t], 0, 0, 0);
      }
    }
  }

  // Sum the waves' tiles; lane (n, g) holds D[4g + i][n], i < 4.
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[((wave * T + t) * 4 + i) * 64 + lane] = acc[t][i];
  __syncthreads();
  const int N = 2 * a.H_r * a.d_r;
  for (int e = threadIdx.x; e < 256 * T; e += kFeThreads) {
    float s = 0.f;
#pragma unroll
    for (int w = 0; w < kFeWaves; ++w) s += red[w * 256 * T + e];
    const int t = e >> 8, i = (e >> 6) & 3, l = e & 63;
    const int b = b0 + 16 * t + 4 * (l >> 4) + i;
    const int nn = l & 15;
    const int f = mat * a.H_r * a.d_r + h * a.d_r + i0 + (nn & 7) + (nn >> 3) * (a.d_r / 2);
    if (b < a.B) a.part[((size_t)split * a.B + b) * N + f] = s;
  }
}

__global__ __launch_bounds__(kFinishThreads) void qk_finish_kernel(FrontArgs a) {
  const int half = a.d_r / 2;
  const int total = a.B * 2 * a.H_r * half;
  const int e = blockIdx.x * kFinishThreads + threadIdx.x;
  if (e >= total) return;
  const int i = e % half;
  const int r = e / half;
  const int h = r % a.H_r;
  const int mat = (r / a.H_r) & 1;
  const int b = r / (2 * a.H_r);
  const int N = 2 * a.H_r * a.d_r;
  const int f = mat * a.H_r * a.d_r + h * a.d_r + i;
  float x = 0.f, y = 0.f;
  for (int s = 0; s < a.ks; ++s) {
    const float* p = a.part + ((size_t)s * a.B + b) * N + f;
    x += p[0];
    y += p[half];
  }
  store_pair(a, mat, b, h, i, x, y, a.theta[i], (float)a.theta[half]);
}

// 17 to 64 sequences, one kernel (qk_full_kernel): a workgroup owns the 16
// features of qk_partial_kernel's tile (dimensions i0..i0+7 of one head and
// their rotary partners) for 16 tokens over the WHOLE hidden dimension; its
// waves take the 128-element steps in turn (the loads of up to CH steps
// issued before the first MFMA), their tiles are summed in LDS in wave order
// (deterministic), and the pairs are rotated and stored in the epilogue: no
// partial sums leave the workgroup.  The token blocks of one feature tile
// are n_tiles = 2 H_r d_r / 16 workgroups apart, a multiple of the 8 XCDs,
// so they run on one XCD and its L2 serves the tile's weight rows to all of
// them after the first read.
constexpr int kFullWaves = 8;
template <int T, int kFullWaves, int CH>
__global__ __launch_bounds__(64 * kFullWaves) void qk_full_kernel(FrontArgs a) {
  constexpr int kFullThreads = 64 * kFullWaves;
  __shared__ float red[kFullWaves * T * 256];
  __shared__ double theta[8];
  __shared__ float mscale;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int tiles_per_head = a.d_r / 16;
  const int per_mat = a.H_r * tiles_per_head;
  const int tile = blockIdx.x;
  const int mat = tile / per_mat;  // 0: Q, 1: K
  const int rem = tile - mat * per_mat;
  const int h = rem / tiles_per_head;
  const int i0 = 8 * (rem - h * tiles_per_head);
  const int b0 = blockIdx.y * 16 * T;
  const int n_steps = a.hidden / kFeStep;

  const int n = lane & 15;
  const int g = lane >> 4;
  const int fbase = h * a.d_r + i0 + (n & 7) + (n >> 3) * (a.d_r / 2);
  const uint16_t* wrow = (mat ? a.w_k : a.w_q) + (size_t)fbase * a.hidden + 8 * g;
  const uint16_t* erow[T];
#pragma unroll
  for (int t = 0; t < T; ++t) {
    const int b = min(b0 + 16 * t + n, a.B - 1);  // rows past B compute a copy, never stored
    const int tok = clampi(a.tokens[b], 0, a.vocab - 1);
    erow[t] = a.emb + (size_t)tok * a.hidden + 8 * g;
  }
  if (wave == 0 && lane < 8) {  // frequencies of this tile's pairs, while the loads fly
    theta[lane] = yarn_theta(a, i0 + lane);
    if (lane == 0) mscale = a.scale > 1.0f ? (float)(0.1 * log((double)a.scale) + 1.0) : 1.0f;
  }

  floatx4 acc[T];
#pragma unroll
  for (int t = 0; t < T; ++t) acc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
  for (int s0 = wave; s0 < n_steps; s0 += kFullWaves * CH) {
    // the loads of CH steps, all issued before the first MFMA (steps past the
    // row re-read its last step and are not accumulated)
    uint4 w[CH][4];
    uint4 e[CH][T][4];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      const size_t off = (size_t)min(s0 + c * kFullWaves, n_steps - 1) * kFeStep;
#pragma unroll
      for (int j = 0; j < 4; ++j) w[c][j] = ldg16(wrow + off + 32 * j);
#pragma unroll
      for (int t = 0; t < T; ++t)
#pragma unroll
        for (int j = 0; j < 4; ++j) e[c][t][j] = ldg16(erow[t] + off + 32 * j);
    }
    __builtin_amdgcn_sched_barrier(0);  // no MFMA (and its wait) moves above a load
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      if (s0 + c * kFullWaves < n_steps) {  // wave-uniform
#pragma unroll
        for (int t = 0; t < T; ++t)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, e[c][t][j]), __builtin_bit_cast(bf16x8, w[c][j]),
                acc[t], 0, 0, 0);
      }
    }
  }

  // lane (n, g) holds D[4g + i][n]: token 16t + 4g + i, feature n of the tile
#pragma unroll
  for (int t = 0; t < T; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[((wave * T + t) * 4 + i) * 64 + lane] = acc[t][i];
  __syncthreads();
  // one thread per (token, pair): the pair's two features summed over the waves
  for (int e = threadIdx.x; e < 16 * T * 8; e += kFullThreads) {
    const int p = e & 7;
    const int tok = e >> 3;  // 0 .. 16T - 1
    const int t = tok >> 4, r = tok & 15;
    const int i = r & 3, gg = r >> 2;
    const int lx = gg * 16 + p, ly = gg * 16 + 8 + p;  // lanes holding features p and p + half
    float x = 0.f, y = 0.f;
#pragma unroll
    for (int w = 0; w < kFullWaves; ++w) {
      x += red[((w * T + t) * 4 + i) * 64 + lx];
      y += red[((w * T + t) * 4 + i) * 64 + ly];
    }
    const int b = b0 + tok;
    if (b < a.B) store_pair(a, mat, b, h, i0 + p, x, y, theta[p], mscale);
  }
}

constexpr int kGvSlab = 512;  // hidden elements per wave slab: 64 lanes x 8

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

// acc + lo(x) * lo(y) + hi(x) * hi(y) for two packed bf16 pairs.
__device__ __forceinline__ float dot2_bf16(uint32_t x, uint32_t y, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, x),
                                         __builtin_bit_cast(bf16x2, y), acc, false);
}

// TB: token rows held per lane (B <= TB; rows past B repeat the last one and
// are never stored).  CH: slabs whose loads are issued together.
template <int TB, int CH>
__global__ __launch_bounds__(kFeThreads) void qk_gemv_kernel(FrontArgs a) {
  __shared__ float red[kFeWaves * 4 * 4 * TB];  // [wave][row][feature][token]
  __shared__ float tot[4 * TB];
  __shared__ double theta[2];
  __shared__ float mscale;

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int half = a.d_r / 2;
  const int tiles_per_head = a.d_r / 4;
  const int per_mat = a.H_r * tiles_per_head;
  const int mat = blockIdx.x / per_mat;  // 0: Q, 1: K
  const int rem = blockIdx.x - mat * per_mat;
  const int h = rem / tiles_per_head;
  const int i0 = 2 * (rem - h * tiles_per_head);
  // features i0, i0 + 1 and their rotary partners i0 + d_r/2, i0 + 1 + d_r/2
  const uint16_t* wm = (mat ? a.w_k : a.w_q) + (size_t)(h * a.d_r + i0) * a.hidden;
  const uint16_t* wr[4] = {wm, wm + a.hidden, wm + (size_t)half * a.hidden,
                           wm + (size_t)(half + 1) * a.hidden};
  const uint16_t* er[TB];
#pragma unroll
  for (int t = 0; t < TB; ++t) {
    const int tok = clampi(a.tokens[min(t, a.B - 1)], 0, a.vocab - 1);
    er[t] = a.emb + (size_t)tok * a.hidden;
  }

  float acc[4][TB];
#pragma unroll
  for (int f = 0; f < 4; ++f)
#pragma unroll
    for (int t = 0; t < TB; ++t) acc[f][t] = 0.f;

  const int n_slabs = (a.hidden + kGvSlab - 1) / kGvSlab;
  for (int s0 = wave; s0 < n_slabs; s0 += kFeWaves * CH) {
    // Loads of the chunk, all unconditional: past the end of the row a lane
    // re-reads the row's last 8 elements and its products are dropped.
    uint4 w[CH][4];
    uint4 e[CH][TB];
    int kk[CH];
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      kk[c] = min(s0 + c * kFeWaves, n_slabs - 1) * kGvSlab + 8 * lane;
      const int kc = min(kk[c], a.hidden - 8);
#pragma unroll
      for (int f = 0; f < 4; ++f) w[c][f] = ldg16(wr[f] + kc);
#pragma unroll
      for (int t = 0; t < TB; ++t) e[c][t] = ldg16(er[t] + kc);
    }
    __builtin_amdgcn_sched_barrier(0);  // every load of the chunk is in flight first
    if (s0 == wave && wave == 0 && lane < 2) {
      theta[lane] = yarn_theta(a, i0 + lane);
      if (lane == 0) mscale = a.scale > 1.0f ? (float)(0.1 * log((double)a.scale) + 1.0) : 1.0f;
    }
#pragma unroll
    for (int c = 0; c < CH; ++c) {
      if (s0 + c * kFeWaves < n_slabs && kk[c] < a.hidden) {
        // v_dot2_f32_bf16: two bf16 products added to the fp32 sum
#pragma unroll
        for (int t = 0; t < TB; ++t)
#pragma unroll
          for (int f = 0; f < 4; ++f) {
            acc[f][t] = dot2_bf16(w[c][f].x, e[c][t].x, acc[f][t]);
            acc[f][t] = dot2_bf16(w[c][f].y, e[c][t].y, acc[f][t]);
            acc[f][t] = dot2_bf16(w[c][f].z, e[c][t].z, acc[f][t]);
            acc[f][t] = dot2_bf16(w[c][f].w, e[c][t].w, acc[f][t]);
          }
      }
    }
  }

  // Reduce: 16-lane rows by DPP (all chains first, so that they interleave),
  // then the 4 rows x 4 waves in LDS.
#pragma unroll
  for (int f = 0; f < 4; ++f)
#pragma unroll
    for (int t = 0; t < TB; ++t) acc[f][t] = row_sum<16>(acc[f][t]);
  if ((lane & 15) == 0) {
#pragma unroll
    for (int f = 0; f < 4; ++f)
#pragma unroll
      for (int t = 0; t < TB; ++t) red[((wave * 4 + (lane >> 4)) * 4 + f) * TB + t] = acc[f][t];
  }
  __syncthreads();
  if (threadIdx.x < 4 * TB) {
    float s = 0.f;
#pragma unroll
    for (int r = 0; r < kFeWaves * 4; ++r) s += red[r * 4 * TB + threadIdx.x];
    tot[threadIdx.x] = s;
  }
  __syncthreads();
  if (threadIdx.x < 2 * TB) {
    const int p = threadIdx.x / TB, t = threadIdx.x - p * TB;
    if (t < a.B)
      store_pair(a, mat, t, h, i0 + p, tot[p * TB + t], tot[(p + 2) * TB + t], theta[p], mscale);
  }
}

struct FrontPlan {
  int ks, steps_per_split;
};

FrontPlan front_plan(const Dims& d, const FrontDims& f) {
  const int n_steps = f.hidden / kFeStep;
  const int n_tiles = 2 * d.H_r * (d.d_r / 16);
  const int row_blocks = (d.B + 63) / 64;
  int ks = (kFeBlocksTarget + n_tiles * row_blocks - 1) / (n_tiles * row_blocks);
  ks = ks < 1 ? 1 : (ks > kFrontMaxSplit ? kFrontMaxSplit : ks);
  ks = ks > n_steps ? n_steps : ks;
  FrontPlan p;
  p.steps_per_split = (n_steps + ks - 1) / ks;
  p.ks = (n_steps + p.steps_per_split - 1) / p.steps_per_split;
  return p;
}

template <int TB>
void launch_gemv(const FrontArgs& a, hipStream_t s) {
  const int grid = 2 * a.H_r * (a.d_r / 4);
  const int n_slabs = (a.hidden + kGvSlab - 1) / kGvSlab;
  const int per_wave = (n_slabs + kFeWaves - 1) / kFeWaves;
  if constexpr (TB <= 4) {
    if (per_wave >= 4) {
      hipLaunchKernelGGL((qk_gemv_kernel<TB, 4>), dim3(grid), dim3(kFeThreads), 0, s, a);
      return;
    }
  }
  if (per_wave >= 2)
    hipLaunchKernelGGL((qk_gemv_kernel<TB, 2>), dim3(grid), dim3(kFeThreads), 0, s, a);
  else
    hipLaunchKernelGGL((qk_gemv_kernel<TB, 1>), dim3(grid), dim3(kFeThreads), 0, s, a);
}

template <int T>
void launch_partial(const FrontArgs& a, dim3 grid, hipStream_t s) {
  // steps per wave; one chunk covers them all when the registers allow
  const int per_wave = (a.steps_per_split + kFeWaves - 1) / kFeWaves;
  if constexpr (T == 1) {
    if (per_wave >= 4) {
      hipLaunchKernelGGL((qk_partial_kernel<T, 4>), grid, dim3(kFeThreads), 0, s, a);
      return;
    }
  }
  if (per_wave >= 2)
    hipLaunchKernelGGL((qk_partial_kernel<T, 2>), grid, dim3(kFeThreads), 0, s, a);
  else
    hipLaunchKernelGGL((qk_partial_kernel<T, 1>), grid, dim3(kFeThreads), 0, s, a);
}

}  // namespace

// Workspace: the frequency table and m, then the partial sums.
static size_t front_table_bytes(const Dims& d) {
  return align_up(sizeof(double) * (size_t)(d.d_r / 2 + 1));
}

size_t front_ws_bytes(const Dims& d) {
  return front_table_bytes(d) +
         align_up(sizeof(float) * (size_t)kFrontMaxSplit * d.B * 2 * d.H_r * d.d_r);
}

hipError_t launch_retrieval_qk(const Dims& d, const FrontDims& f, const int32_t* tokens,
                               const int32_t* pos, const uint16_t* emb, const uint16_t* w_q,
                               const uint16_t* w_k, uint16_t* q_r, uint16_t* k_r, void* ws,
                               hipStream_t s) {
  const FrontPlan p = front_plan(d, f);
  FrontArgs a;
  a.tokens = tokens;
  a.pos = pos;
  a.emb = emb;
  a.w_q = w_q;
  a.w_k = w_k;
  a.q_r = q_r;
  a.k_r = k_r;
  a.theta = static_cast<double*>(ws);
  a.part = reinterpret_cast<float*>(static_cast<char*>(ws) + front_table_bytes(d));
  a.kr_stride_b = d.kr_stride_b;
  a.B = d.B;
  a.vocab = f.vocab;
  a.hidden = f.hidden;
  a.H_r = d.H_r;
  a.d_r = d.d_r;
  a.L_cap = d.L_cap;
  a.ks = p.ks;
  a.steps_per_split = p.steps_per_split;
  a.base = f.base;
  a.scale = f.scale;
  a.alpha = f.alpha;
  a.beta = f.beta;
  a.orig_ctx = f.orig_ctx;
  if (d.B <= 16) {  // one kernel, whole hidden dimension per workgroup
    if (d.B == 1) launch_gemv<1>(a, s);
    else if (d.B == 2) launch_gemv<2>(a, s);
    else if (d.B <= 4) launch_gemv<4>(a, s);
    else if (d.B <= 8) launch_gemv<8>(a, s);
    else launch_gemv<16>(a, s);
    return hipGetLastError();
  }
  const int n_tiles = 2 * d.H_r * (d.d_r / 16);
  if (d.B <= 64) {  // one kernel: 16 tokens and 16 features per workgroup, whole rows
    const dim3 grid(n_tiles, (d.B + 15) / 16);
    const int per_wave = (f.hidden / kFeStep + kFullWaves - 1) / kFullWaves;
    if (per_wave >= 4)
      hipLaunchKernelGGL((qk_full_kernel<1, kFullWaves, 4>), grid, dim3(64 * kFullWaves), 0, s, a);
    else if (per_wave >= 2)
      hipLaunchKernelGGL((qk_full_kernel<1, kFullWaves, 2>), grid, dim3(64 * kFullWaves), 0, s, a);
    else
      hipLaunchKernelGGL((qk_full_kernel<1, kFullWaves, 1>), grid, dim3(64 * kFullWaves), 0, s, a);
    return hipGetLastError();
  }
  launch_partial<4>(a, dim3(n_tiles * p.ks, (d.B + 63) / 64), s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int total = d.B * d.H_r * d.d_r;  // B * 2 * H_r * d_r/2 pairs
  hipLaunchKernelGGL(qk_finish_kernel, dim3((total + kFinishThreads - 1) / kFinishThreads),
                     dim3(kFinishThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace spec
