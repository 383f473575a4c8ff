// Sparse GQA decode attention on gfx950 (SpeContext Eq. 1 over the selected
// tokens; Sec. 4.3 "Support for GQA": the G query heads of a group share one
// KV head, which is read directly -- no repeat_kv copy).
//
// Split-K flash decode.  One wavefront owns a work item (layer, sequence,
// KV head g, split of the selection) and walks it in chunks of 64 selected
// tokens:
//  * Q.K^T on the matrix cores: v_mfma_f32_16x16x32_bf16 with A = the G
//    query heads of the group (rows >= G are zero) and B = 16 selected K rows,
//    each lane feeding one 16-byte slice of one row straight from HBM, so K
//    needs no LDS staging and no bf16->fp32 conversion.  The useful fraction
//    of the tile is G/16, irrelevant here: the op is HBM-bound by two orders
//    of magnitude.
//  * online softmax in log2 units (the scale and log2(e) are folded into one
//    multiply), P and the rescale factors go through a 4 KB LDS slice;
//  * P.V on the vector ALUs: lane (q, c) owns the 8 dims 8c..8c+7 of every
//    4th token of the chunk, accumulating G x 8 fp32 values; V rows arrive as
//    16-byte loads, four full 256-byte rows per load instruction.
// A second kernel merges the per-split (max, sum, acc) partials with a
// log-sum-exp combine and writes fp32 out and lse.
#include "device_common.h"
#include "internal.h"

namespace spec {
namespace {

constexpr int kWaves = 4;   // wavefronts per workgroup
constexpr int kChunk = 64;  // selected tokens per inner step
constexpr int kD = 128;     // head dimension

struct AttnArgs {
  const uint16_t* q;      // [n_layers][B][H_q][d]
  const uint16_t* k;      // indexed: cache; compact: [n_layers][B][k_max][H_kv][d]
  const uint16_t* v;
  const int32_t* idx;     // [B][k_max] (indexed mode)
  const int32_t* counts;  // [B]
  float* part_acc;        // [n_layers*B][n_split][H_q][d]
  float* part_ml;         // [n_layers*B][n_split][H_q][2]
  int64_t stride_layer;   // elements between layers (indexed mode)
  int64_t stride_b;       // elements between sequences (indexed mode)
  int B, H_q, H_kv, k_max, L_cap, n_split, split_tokens, n_items;
  float scale_log2;       // scale * log2(e)
};

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int G, bool INDEXED>
__global__ __launch_bounds__(kWaves * 64) void attn_split_kernel(AttnArgs a) {
  __shared__ float lds[kWaves][kChunk * G + 16];  // P[token][head], then alpha[G]
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int item = blockIdx.x * kWaves + wave;
  if (item >= a.n_items) return;  // uniform per wavefront; no block barriers below
  const int g = item % a.H_kv;
  const int rest = item / a.H_kv;
  const int split = rest % a.n_split;
  const int lb = rest / a.n_split;  // layer * B + b
  const int b = lb % a.B;
  const int layer = lb / a.B;
  const int count = clampi(a.counts[b], 0, a.k_max);
  const int j0 = split * a.split_tokens;
  if (j0 >= count) return;
  const int j1 = min(j0 + a.split_tokens, count);

  const int64_t rs = (int64_t)a.H_kv * kD;  // elements per token row
  const uint16_t* kb;
  const uint16_t* vb;
  if (INDEXED) {
    const int64_t off = (int64_t)layer * a.stride_layer + (int64_t)b * a.stride_b + g * kD;
    kb = a.k + off;
    vb = a.v + off;
  } else {
    const int64_t off = (int64_t)lb * a.k_max * rs + g * kD;
    kb = a.k + off;
    vb = a.v + off;
  }
  const int32_t* idx_b = INDEXED ? a.idx + (size_t)b * a.k_max : nullptr;

  const int r16 = lane & 15;  // MFMA row/column index of this lane
  const int kg = lane >> 4;   // MFMA k-group of this lane
  // A operand: query head g*G + r16, dims 32s + 8kg .. +8 (zero rows >= G).
  bf16x8 qf[4];
  {
    const uint16_t* qp = a.q + ((size_t)lb * a.H_q + g * G + (r16 < G ? r16 : 0)) * kD + 8 * kg;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      uint4 w = r16 < G ? ldg16(qp + 32 * s) : make_uint4(0, 0, 0, 0);
      qf[s] = __builtin_bit_cast(bf16x8, w);
    }
  }

  float m_run[4], l_run[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    m_run[i] = -INFINITY;
    l_run[i] = 0.f;
  }
  float acc[G][8];
#pragma unroll
  for (int m = 0; m < G; ++m)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[m][e] = 0.f;

  float* P = lds[wave];
  const int vq = lane >> 4;  // P.V: token phase of this lane
  const int vc = lane & 15;  // P.V: 8-dim column block of this lane

  for (int c0 = j0; c0 < j1; c0 += kChunk) {
    // Row of selected token c0 + lane (masked tokens read row 0).
    const int jl = c0 + lane;
    int myrow = 0;
    if (jl < j1) myrow = INDEXED ? clampi(idx_b[jl], 0, a.L_cap - 1) : jl;

    uint4 kraw[4][4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int row = __shfl(myrow, 16 * t + r16);
      const uint16_t* p = kb + (int64_t)row * rs + 8 * kg;
#pragma unroll
      for (int s = 0; s < 4; ++s) kraw[t][s] = ldg16(p + 32 * s);
    }
    uint4 vraw[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int row = __shfl(myrow, vq + 4 * r);
      vraw[r] = ldg16(vb + (int64_t)row * rs + 8 * vc);
    }

    // S = Q K^T for 4 tiles of 16 tokens; lane holds S[head 4kg+i][token r16].
    float sv[4][4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      floatx4 sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s)
        sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(qf[s], __builtin_bit_cast(bf16x8, kraw[t][s]),
                                                       sacc, 0, 0, 0);
      const bool valid = c0 + 16 * t + r16 < j1;
#pragma unroll
      for (int i = 0; i < 4; ++i) sv[t][i] = valid ? sacc[i] * a.scale_log2 : -INFINITY;
    }
    float alpha[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float mx = fmaxf(fmaxf(sv[0][i], sv[1][i]), fmaxf(sv[2][i], sv[3][i]));
#pragma unroll
      for (int off = 1; off < 16; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off, 16));
      const float mn = fmaxf(m_run[i], mx);
      alpha[i] = exp2f(m_run[i] - mn);
      float ls = 0.f;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        sv[t][i] = exp2f(sv[t][i] - mn);
        ls += sv[t][i];
      }
      l_run[i] = l_run[i] * alpha[i] + ls;
      m_run[i] = mn;
    }
    // P (and alpha) to LDS for the P.V lane layout.
    if (4 * kg < G) {
#pragma unroll
      for (int t = 0; t < 4; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (4 * kg + i < G) P[(16 * t + r16) * G + 4 * kg + i] = sv[t][i];
      if (r16 == 0) {
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (4 * kg + i < G) P[kChunk * G + 4 * kg + i] = alpha[i];
      }
    }
    wave_sync_lds();

#pragma unroll
    for (int m = 0; m < G; ++m) {
      const float al = P[kChunk * G + m];
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[m][e] *= al;
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      float vf[8];
      unpack8(vraw[r], vf);
      const float* pr = P + (vq + 4 * r) * G;
#pragma unroll
      for (int m = 0; m < G; ++m) {
        const float pm = pr[m];
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[m][e] = fmaf(pm, vf[e], acc[m][e]);
      }
    }
    wave_sync_lds();  // P is rewritten by the next chunk
  }

  // Row sums over the 16 token lanes; accumulators over the 4 token phases.
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int off = 1; off < 16; off <<= 1) l_run[i] += __shfl_xor(l_run[i], off, 16);
#pragma unroll
  for (int m = 0; m < G; ++m)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      acc[m][e] += __shfl_xor(acc[m][e], 16);
      acc[m][e] += __shfl_xor(acc[m][e], 32);
    }

  const size_t prow = ((size_t)lb * a.n_split + split) * a.H_q + (size_t)g * G;
  if (vq == 0) {
#pragma unroll
    for (int m = 0; m < G; ++m) {
      float4* dst = reinterpret_cast<float4*>(a.part_acc + (prow + m) * kD + 8 * vc);
      dst[0] = make_float4(acc[m][0], acc[m][1], acc[m][2], acc[m][3]);
      dst[1] = make_float4(acc[m][4], acc[m][5], acc[m][6], acc[m][7]);
    }
  }
  if (r16 == 0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if (4 * kg + i < G) {
        float* ml = a.part_ml + (prow + 4 * kg + i) * 2;
        ml[0] = m_run[i];
        ml[1] = l_run[i];
      }
    }
  }
}

struct CombineArgs {
  const float* part_acc;
  const float* part_ml;
  const int32_t* counts;
  float* out;  // [n_layers*B][H_q][d]
  float* lse;  // [n_layers*B][H_q] or null
  int B, H_q, k_max, n_split, split_tokens;
};

// One workgroup per (layer*B + b, group of 8 heads); thread = (head, 4 dims).
__global__ __launch_bounds__(256) void attn_combine_kernel(CombineArgs a) {
  const int lb = blockIdx.x;
  const int h = blockIdx.y * 8 + (threadIdx.x >> 5);
  const int d4 = threadIdx.x & 31;
  if (h >= a.H_q) return;
  const int b = lb % a.B;
  const int count = clampi(a.counts[b], 0, a.k_max);
  const int ns = (count + a.split_tokens - 1) / a.split_tokens;
  float4* o = reinterpret_cast<float4*>(a.out + ((size_t)lb * a.H_q + h) * kD) + d4;
  if (ns == 0) {
    *o = make_float4(0.f, 0.f, 0.f, 0.f);
    if (a.lse && d4 == 0) a.lse[(size_t)lb * a.H_q + h] = -INFINITY;
    return;
  }
  const size_t base = (size_t)lb * a.n_split * a.H_q + h;  // row of split 0
  float M = -INFINITY;
  for (int s = 0; s < ns; ++s) M = fmaxf(M, a.part_ml[(base + (size_t)s * a.H_q) * 2]);
  float L = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s = 0; s < ns; ++s) {
    const size_t row = base + (size_t)s * a.H_q;
    const float w = exp2f(a.part_ml[row * 2] - M);
    L += a.part_ml[row * 2 + 1] * w;
    const float4 p = reinterpret_cast<const float4*>(a.part_acc + row * kD)[d4];
    acc.x += p.x * w;
    acc.y += p.y * w;
    acc.z += p.z * w;
    acc.w += p.w * w;
  }
  const float inv = 1.f / L;
  *o = make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
  if (a.lse && d4 == 0) a.lse[(size_t)lb * a.H_q + h] = (M + log2f(L)) * kLn2;
}

template <bool INDEXED>
void launch_split(int G, dim3 grid, hipStream_t s, const AttnArgs& a) {
  switch (G) {
    case 1: attn_split_kernel<1, INDEXED><<<grid, kWaves * 64, 0, s>>>(a); break;
    case 2: attn_split_kernel<2, INDEXED><<<grid, kWaves * 64, 0, s>>>(a); break;
    case 4: attn_split_kernel<4, INDEXED><<<grid, kWaves * 64, 0, s>>>(a); break;
    case 8: attn_split_kernel<8, INDEXED><<<grid, kWaves * 64, 0, s>>>(a); break;
    default: attn_split_kernel<16, INDEXED><<<grid, kWaves * 64, 0, s>>>(a); break;
  }
}

}  // namespace

int attn_split_tokens(const Dims& d) {
  // Longest split (fewest partials to write and merge) that still yields at
  // least 2048 wavefront work items to spread over the 256 compute units.
  const int64_t base = (int64_t)d.n_layers * d.B * d.H_kv;
  const int cand[3] = {512, 256, 128};
  for (int i = 0; i < 3; ++i) {
    const int64_t ns = (d.k_max + cand[i] - 1) / cand[i];
    if (base * ns >= 2048) return cand[i];
  }
  return 64;
}

hipError_t launch_attn(const Dims& d, const uint16_t* q, const uint16_t* k,
                       const uint16_t* v, const int32_t* idx, const int32_t* counts,
                       float* out, float* lse, void* ws, hipStream_t s) {
  const int split = attn_split_tokens(d);
  const int n_split = attn_n_split(d);
  const size_t rows = (size_t)d.n_layers * d.B * n_split * d.H_q;
  float* part_acc = static_cast<float*>(ws);
  float* part_ml = reinterpret_cast<float*>(static_cast<char*>(ws) +
                                            align_up(sizeof(float) * rows * d.d));
  const int64_t n_items = (int64_t)d.n_layers * d.B * n_split * d.H_kv;
  AttnArgs a{q, k, v, idx, counts, part_acc, part_ml, d.kv_stride_layer, d.kv_stride_b,
             d.B, d.H_q, d.H_kv, d.k_max, d.L_cap, n_split, split, (int)n_items,
             d.scale * kLog2e};
  const dim3 grid((unsigned)((n_items + kWaves - 1) / kWaves));
  if (idx)
    launch_split<true>(d.G, grid, s, a);
  else
    launch_split<false>(d.G, grid, s, a);
  CombineArgs c{part_acc, part_ml, counts, out, lse, d.B, d.H_q, d.k_max, n_split, split};
  const dim3 g2(d.n_layers * d.B, (d.H_q + 7) / 8);
  attn_combine_kernel<<<g2, 256, 0, s>>>(c);
  return hipGetLastError();
}

}  // namespace spec
