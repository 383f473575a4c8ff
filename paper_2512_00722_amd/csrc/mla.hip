// Sparse decode attention of an MLA model (Sec. 4.3, "Support for MLA"): the
// cache holds one latent row per token -- the latent c (d_c = 512) followed by
// the rotary key shared by all heads (d_rope = 64) -- and only the selected
// rows are raised to per-head keys [W_UK[h] c ; k_rope] and values W_UV[h] c.
//
// The kernels compute the same attention in the absorbed form, which never
// materialises a per-head key or value:
//   q~_h = W_UK[h]^T q_nope_h  (and q_rope_h appended), so that
//   q_h . key_{h,j} = q~_h . [c_j ; k_rope_j];
//   o_h = W_UV[h] (sum_j p_hj c_j), since the weights p_hj sum to one.
// All H heads then read the same selected latent rows (multi-query
// attention with 576-wide keys and 512-wide values).  Three kernels:
//
//  1. mla_absorb_kernel: one wavefront per (layer, head) streams W_UK[h]
//     (d_nope rows of d_c) once for every sequence, forms q~ with
//     v_dot2_f32_bf16 (exact products, fp32 sums) and stores it as a bf16
//     high part and a bf16 low part (q~ - high), so that it reaches the
//     matrix cores to ~2^-17; the rotary part is copied as is (already bf16)
//     and the scale is applied to the fp32 logits.
//  2. mla_attn_kernel: one workgroup per CU, four wavefronts; a work unit is
//     (layer, sequence, split of the selection, group of 64 heads).  Per
//     32-token chunk the selected latent rows go from HBM straight into LDS
//     (no registers; four stages, so three chunks stream in during this
//     chunk's math), and every wavefront -- 16 heads -- runs
//       S^T = C Q~^T  on v_mfma_f32_16x16x32_bf16 (A = 16 latent rows from
//                     LDS, B = q~ of 16 heads, resident in registers: two
//                     MFMAs per k-step on the latent part, high and low),
//       online softmax in log2 units per head,
//       O^T += C^T P^T (A = latent columns read transposed from LDS with
//                     ds_read_b64_tr_b16, B = P as a bf16 high + low pair,
//                     both truncated: 2^-14 relative).
//     It leaves (max, sum, acc) per (unit, head) in the workspace.  A wave
//     holds q~ of its heads (136 registers, in AGPRs: only ever an MFMA
//     operand) and their latent accumulator (128, in VGPRs: this file is
//     built with MFMA results in VGPRs, so that the rare rescale of the
//     accumulators needs no copies): a register file of 512 fits 16 heads,
//     not 32, so 128 heads take two workgroups.  Their work units are
//     numbered 8 apart, which puts them on the same XCD (workgroups are
//     dealt to the 8 XCDs in turn) at the same time: the second reads the
//     latent rows from that XCD's L2.
//  3. mla_out_kernel: one workgroup per (layer, head) merges the splits of
//     every sequence into the latent output o~ (log-sum-exp), splits it into
//     bf16 high + low parts in LDS and applies W_UV[h] on the matrix cores
//     (A = 16 rows of W_UV streamed from HBM, B = o~ of up to 16 sequences),
//     writing out and lse.
#include "device_common.h"
#include "internal.h"

namespace spec {
namespace {

constexpr int kDC = 512;             // latent width
constexpr int kDR = 64;              // rotary key width
constexpr int kDK = kDC + kDR;       // key width of the latent row
constexpr int kDN = 128;             // per-head no-position query width
constexpr int kDVo = 128;            // per-head value width
constexpr int kMWaves = 4;           // wavefronts per workgroup
constexpr int kMThreads = 64 * kMWaves;
constexpr int kMChunk = 32;          // selected tokens per inner step
constexpr int kQSteps = kDK / 32;    // k-steps of S^T = C Q~^T
constexpr int kLSteps = kDC / 32;    // k-steps on the latent part (high + low)
constexpr int kQT = 2 * kDC + kDR;   // absorbed query row: high, low, rotary
constexpr int kVBlocks = kDC / 16;   // 16-dim blocks of O^T
constexpr int kMMaxSplit = 2048;     // longest split (tokens per work unit)
constexpr int kMMinSplit = 256;
constexpr int kMMaxSplitCount = 16;  // splits per (layer, sequence); the merge holds 16 weights
constexpr float kLazy = 8.f;         // log2 headroom of the lazy softmax reference

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

struct MlaArgs {
  const uint16_t* q;       // [n_layers][B][H][d_nope + d_rope]
  const uint16_t* ckv;     // latent rows [n_layers][B][L_cap][576] (strides below)
  const uint16_t* w_uk;    // [n_layers][H][d_nope][d_c]
  const uint16_t* w_uv;    // [n_layers][H][d_v][d_c]
  const int32_t* idx;      // [B][k_max]
  const int32_t* counts;   // [B]
  uint16_t* qt;            // workspace: [n_layers][B][H][2 d_c + d_rope] absorbed queries
  float* part_acc;         // workspace: [n_layers * B][n_split][H][d_c]
  float* part_ml;          // workspace: [n_layers * B][n_split][H][2]
  float* out;              // [n_layers][B][H][d_v]
  float* lse;              // [n_layers][B][H] or null
  int64_t stride_layer, stride_b;  // elements of ckv
  int B, H, k_max, L_cap, n_layers, n_split, split_tokens, n_units, n_hg, n_items;
  float scale_log2;        // scale * log2(e)
};

__device__ __forceinline__ uint32_t f2bf_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// 8 values -> bf16 high part and bf16 low part (value - high), packed.
__device__ __forceinline__ void split8(const float* p, uint4& hi, uint4& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t h0 = f2bf_rne(p[2 * j]), h1 = f2bf_rne(p[2 * j + 1]);
    const uint32_t l0 = f2bf_rne(p[2 * j] - __uint_as_float(h0 << 16));
    const uint32_t l1 = f2bf_rne(p[2 * j + 1] - __uint_as_float(h1 << 16));
    h[j] = h0 | (h1 << 16);
    l[j] = l0 | (l1 << 16);
  }
  hi = make_uint4(h[0], h[1], h[2], h[3]);
  lo = make_uint4(l[0], l[1], l[2], l[3]);
}

// 8 values -> bf16 high part (truncated) and bf16 low part (the exact fp32
// remainder, truncated), packed: the pair holds each value to 2^-14
// relative, in six instructions per two values where the rounded split
// takes about twenty.
__device__ __forceinline__ void split8_trunc(const float* p, uint4& hi, uint4& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t u0 = __float_as_uint(p[2 * j]), u1 = __float_as_uint(p[2 * j + 1]);
    const float r0 = p[2 * j] - __uint_as_float(u0 & 0xffff0000u);
    const float r1 = p[2 * j + 1] - __uint_as_float(u1 & 0xffff0000u);
    h[j] = __builtin_amdgcn_perm(u1, u0, 0x07060302u);  // high halves of u0 (low), u1 (high)
    l[j] = __builtin_amdgcn_perm(__float_as_uint(r1), __float_as_uint(r0), 0x07060302u);
  }
  hi = make_uint4(h[0], h[1], h[2], h[3]);
  lo = make_uint4(l[0], l[1], l[2], l[3]);
}

// max / sum over the four lanes {l, l^16, l^32, l^48} (one head's lanes).
__device__ __forceinline__ float xg_max(float v) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float xg_sum(float v) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Transposing LDS read: within each 16-lane group, lane i receives element
// (i & 3) of the 8-byte chunks read by lanes (i >> 2) + 4j, j = 0..3.
__device__ __forceinline__ bf16x4 lds_read_tr(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (__attribute__((address_space(3))) bf16x4*)(p));
}

// ---------------------------------------------------------------------------
// 1. q~ = [W_UK[h]^T q_nope (high, low) ; q_rope]
// ---------------------------------------------------------------------------
// One wavefront per (layer, head): lane l owns latent dims 8l..8l+7 and walks
// the d_nope rows of W_UK[h] in batches of 16 (one 1 KiB row per load
// instruction), two batches in flight: the next batch is requested before
// this one is used.  Rows n and n+1 are paired per latent dim with a byte
// permute and meet the query pair (q[n], q[n+1]) -- the input's own 32-bit
// words, staged in LDS -- in one v_dot2_f32_bf16 (exact products, fp32
// sum): 64 dot products and 8 permutes per row pair for 8 sequences, where
// unpacking and fp32 FMAs took twice as many instructions.  Up to TB
// sequences per pass.
constexpr int kAbsBatch = 8;
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float dot2_bf16(uint32_t x, uint32_t y, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, x),
                                         __builtin_bit_cast(bf16x2, y), acc, false);
}

template <int TB>
__global__ __launch_bounds__(64) void mla_absorb_kernel(MlaArgs a) {
  __shared__ __align__(16) uint32_t qs2[TB][kDN / 2];  // (q[2p], q[2p+1]) as bf16 pairs
  const int lane = threadIdx.x;
  const int layer = blockIdx.x / a.H;
  const int h = blockIdx.x - layer * a.H;
  const uint16_t* w = a.w_uk + ((size_t)layer * a.H + h) * kDN * kDC + 8 * lane;
  auto load = [&](uint4 (&wr)[kAbsBatch], int bt) {
#pragma unroll
    for (int i = 0; i < kAbsBatch; ++i) wr[i] = ldg16_stream(w + (size_t)(bt * kAbsBatch + i) * kDC);
  };
  for (int b0 = 0; b0 < a.B; b0 += TB) {
    uint4 wa[kAbsBatch], wb[kAbsBatch];
    load(wa, 0);
    __syncthreads();  // the previous pass is done with qs2
    // this head's no-position queries of sequences b0 .. b0+TB-1: four pairs a load
    for (int e = lane; e < TB * (kDN / 8); e += 64) {
      const int t = e / (kDN / 8), n8 = e - t * (kDN / 8);
      const int b = min(b0 + t, a.B - 1);
      *reinterpret_cast<uint4*>(&qs2[t][4 * n8]) =
          ldg16(a.q + (((size_t)layer * a.B + b) * a.H + h) * (kDN + kDR) + 8 * n8);
    }
    __syncthreads();
    float acc[TB][8];
#pragma unroll
    for (int t = 0; t < TB; ++t)
#pragma unroll
      for (int j = 0; j < 8; ++j) acc[t][j] = 0.f;
    auto use = [&](const uint4 (&wr)[kAbsBatch], int bt) {
#pragma unroll
      for (int i = 0; i < kAbsBatch / 2; ++i) {
        const uint32_t* x = reinterpret_cast<const uint32_t*>(&wr[2 * i]);      // row n
        const uint32_t* y = reinterpret_cast<const uint32_t*>(&wr[2 * i + 1]);  // row n+1
        uint32_t wp[8];  // (W[n][c], W[n+1][c]) for this lane's 8 latent dims
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          wp[2 * j] = __builtin_amdgcn_perm(y[j], x[j], 0x05040100u);
          wp[2 * j + 1] = __builtin_amdgcn_perm(y[j], x[j], 0x07060302u);
        }
#pragma unroll
        for (int t = 0; t < TB; ++t) {
          const uint32_t qp = qs2[t][bt * (kAbsBatch / 2) + i];
#pragma unroll
          for (int c = 0; c < 8; ++c) acc[t][c] = dot2_bf16(wp[c], qp, acc[t][c]);
        }
      }
    };
    // the scheduling barriers keep the order as written: a batch's loads are
    // issued before the other batch is used, so that they are in flight
    // during it, and a refill comes after the last use of its buffer
#pragma unroll 1
    for (int bt = 0; bt < kDN / kAbsBatch; bt += 2) {
      load(wb, bt + 1);
      __builtin_amdgcn_sched_barrier(0);
      use(wa, bt);
      __builtin_amdgcn_sched_barrier(0);
      if (bt + 2 < kDN / kAbsBatch) load(wa, bt + 2);
      __builtin_amdgcn_sched_barrier(0);
      use(wb, bt + 1);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int t = 0; t < TB; ++t) {
      const int b = b0 + t;
      if (b >= a.B) break;
      uint16_t* dst = a.qt + (((size_t)layer * a.B + b) * a.H + h) * kQT;
      uint4 hi, lo;
      split8(acc[t], hi, lo);
      *reinterpret_cast<uint4*>(dst + 8 * lane) = hi;
      *reinterpret_cast<uint4*>(dst + kDC + 8 * lane) = lo;
      if (lane < kDR / 8) {  // the rotary part, unchanged
        const uint16_t* src = a.q + (((size_t)layer * a.B + b) * a.H + h) * (kDN + kDR) + kDN;
        *reinterpret_cast<uint4*>(dst + 2 * kDC + 8 * lane) = ldg16(src + 8 * lane);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// 2. latent attention over the selected rows
// ---------------------------------------------------------------------------
// LDS stage of 32 selected tokens, filled straight from HBM by
// global_load_lds_dwordx4 (lane l of an instruction lands at base + 16 l):
//  * latent region: one instruction per token (its 512 latent dims, 1 KiB),
//    rows 1056 bytes apart (32 bytes apart modulo 256: the transposed reads
//    of four rows and the row reads of sixteen spread over the banks);
//  * rotary region: one instruction per 8 tokens (8 x 128 bytes, packed);
//    16-byte piece p of token m sits in slot p ^ (m & 7) of its row.
// Four stages rotate: chunk c is read while chunks c+1 .. c+3 stream in (one
// CU keeps ~100 KiB in flight).  The global-to-LDS loads are issued from
// inline assembly: the compiler, which cannot tell that the stage being read
// is not the one being filled, would otherwise wait for every pending load
// before each LDS read, serialising the ring.  The kernel does the waiting
// itself: a chunk is handed over by an explicit vector-memory count wait
// (loads retire in issue order) and a bare barrier, with compiler-only
// memory barriers around it (a workgroup fence would also wait for every
// pending load).  Nothing else in the kernel uses M0.
constexpr int kLPitch = kDC + 16;                   // latent row pitch (elements)
constexpr int kStageLat = kMChunk * kLPitch;        // elements
constexpr int kStage = kStageLat + kMChunk * kDR;   // elements
constexpr int kStages = 4;
constexpr int kAhead = kStages - 1;  // chunks requested ahead of the one being read
constexpr int kLoadsPerChunk = kMChunk / kMWaves + 1;  // per wavefront: 8 rows + 1 rotary group
static_assert(kMChunk == 8 * kMWaves, "one rotary group of 8 tokens per wavefront");

// s_waitcnt immediates (gfx9 encoding: vmcnt[3:0], expcnt[6:4], lgkmcnt[11:8],
// vmcnt[5:4] in bits [15:14]): wait for the vector-memory count only.
constexpr int waitcnt_vm(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// Global-to-LDS copy of 16 bytes per lane: lane l's bytes land at LDS
// address lds + 16 l (M0 holds the wave-uniform base).  The compiler reserves
// M0 and warns about the clobber; no instruction it generates in this file
// uses M0, which tests/test_isa_cpu.py checks on the generated assembly.
__device__ __forceinline__ void load_to_lds(const void* g, const void* lds) {
  const uint32_t base = (uint32_t)(uintptr_t)lds;
  asm volatile("s_mov_b32 m0, %0\n\tglobal_load_lds_dwordx4 %1, off"
               :
               : "s"(__builtin_amdgcn_readfirstlane(base)), "v"(g)
               : "memory", "m0");
}

// HT: 16-head tiles per wavefront.
template <int HT>
__global__ __launch_bounds__(kMThreads) __attribute__((amdgpu_waves_per_eu(1)))
void mla_attn_kernel(MlaArgs a) {
  __shared__ __align__(16) uint16_t cbuf[kStages * kStage];
  __shared__ int rows[kMMaxSplit + kStages * kMChunk];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int r16 = lane & 15;  // MFMA column: a head of the tile; row: a token of a C tile
  const int kg = lane >> 4;   // MFMA k-group

  for (int item = blockIdx.x; item < a.n_items; item += gridDim.x) {
    // items 8 n_hg q + 8 hg + r: unit 8q + r, head group hg
    const int hg = (item >> 3) % a.n_hg;
    const int unit = item / (8 * a.n_hg) * 8 + (item & 7);
    if (unit >= a.n_units) continue;  // uniform per workgroup
    const int split = unit % a.n_split;
    const int lb = unit / a.n_split;  // layer * B + b
    const int b = lb % a.B;
    const int layer = lb / a.B;
    const int count = clampi(a.counts[b], 0, a.k_max);
    const int j0 = split * a.split_tokens;
    const int n_tok = max(0, min(a.split_tokens, count - j0));
    // rows of the selection, then padding (row 0) for the chunks the
    // pipeline requests past the end
    const int n_pad = (n_tok + kMChunk - 1) / kMChunk * kMChunk + kAhead * kMChunk;

    __syncthreads();  // the previous unit is done with rows and every stage
    for (int j = tid; j < n_pad; j += kMThreads)
      rows[j] = j < n_tok ? clampi(a.idx[(size_t)b * a.k_max + j0 + j], 0, a.L_cap - 1) : 0;

    // q~ of this wavefront's heads (B operand): head
    // 64 hg + 16 (HT wave + ht) + r16, dims 32s + 8kg .. +8.
    const int head0 = 64 * HT * hg + 16 * HT * wave;
    uint4 qh[HT][kQSteps], ql[HT][kLSteps];  // high parts (then rotary), low parts
#pragma unroll
    for (int ht = 0; ht < HT; ++ht) {
      const uint16_t* qp = a.qt + ((size_t)lb * a.H + head0 + 16 * ht + r16) * kQT + 8 * kg;
#pragma unroll
      for (int s = 0; s < kLSteps; ++s) {
        qh[ht][s] = ldg16(qp + 32 * s);
        ql[ht][s] = ldg16(qp + kDC + 32 * s);
      }
#pragma unroll
      for (int s = kLSteps; s < kQSteps; ++s) qh[ht][s] = ldg16(qp + kDC + 32 * s);
    }
    // q~ in registers before the ring starts: the compiler, which does not
    // count the global-to-LDS loads, would otherwise wait for q~ inside the
    // chunk loop with counts that also drain the chunks in flight
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();  // rows staged

    const uint16_t* cb = a.ckv + (int64_t)layer * a.stride_layer + (int64_t)b * a.stride_b;
    // This wavefront's share of chunk cc: latent rows 8 wave .. 8 wave + 7
    // and the rotary group of the same rows.
    // The row indices are read from LDS before the first load is issued:
    // each load's memory clobber would otherwise keep the next index read
    // behind it, one LDS round trip per row.
    auto issue = [&](int cc, int st) {
      uint16_t* base = cbuf + st * kStage;
      constexpr int kRows = kMChunk / kMWaves;
      int ri[kRows];
#pragma unroll
      for (int r = 0; r < kRows; ++r) ri[r] = rows[cc + kRows * wave + r];
      const int m = 8 * wave + (lane >> 3);
      const int rm = rows[cc + m];
#pragma unroll
      for (int r = 0; r < kRows; ++r)
        load_to_lds(cb + (int64_t)ri[r] * kDK + 8 * lane, base + (kRows * wave + r) * kLPitch);
      const int piece = (lane & 7) ^ (m & 7);
      load_to_lds(cb + (int64_t)rm * kDK + kDC + 8 * piece, base + kStageLat + 8 * kDR * wave);
    };

    float m_run[HT], l_run[HT];
    floatx4 acc[HT][kVBlocks];  // O^T[16db + 4kg + i][head r16 of tile ht]
#pragma unroll
    for (int ht = 0; ht < HT; ++ht) {
      m_run[ht] = -INFINITY;
      l_run[ht] = 0.f;
#pragma unroll
      for (int db = 0; db < kVBlocks; ++db) acc[ht][db] = floatx4{0.f, 0.f, 0.f, 0.f};
    }

    if (n_tok > 0) {
#pragma unroll
      for (int i = 0; i < kAhead; ++i) issue(i * kMChunk, i);
    }
    for (int c = 0; c < n_tok; c += kMChunk) {
      const int ci = c / kMChunk;
      // this wavefront's loads of chunk c are done (those of the later
      // chunks may not be), then every wavefront's: the stage is complete,
      // and the stage of chunk c-1 is free for chunk c+kAhead
      __builtin_amdgcn_s_waitcnt(waitcnt_vm((kAhead - 1) * kLoadsPerChunk));
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      issue(c + kAhead * kMChunk, (ci + kAhead) % kStages);
      const uint16_t* C = cbuf + (ci % kStages) * kStage;
      const uint16_t* R = C + kStageLat;

      // S^T tiles: lane holds S[head r16][token 16t + 4kg + i].
      floatx4 sacc[HT][2];
#pragma unroll
      for (int ht = 0; ht < HT; ++ht) {
        sacc[ht][0] = floatx4{0.f, 0.f, 0.f, 0.f};
        sacc[ht][1] = floatx4{0.f, 0.f, 0.f, 0.f};
      }
      // Reads run ahead: the A operands of steps s+1 .. s+3 are read from LDS
      // while the MFMAs of step s run (the scheduling barriers keep the
      // compiler from hoisting every read, which would need ~150 more
      // registers).
      auto read_a = [&](int s, uint4 (&ca)[2]) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const int m = 16 * t + r16;
          ca[t] = s < kLSteps
                      ? *reinterpret_cast<const uint4*>(C + m * kLPitch + 32 * s + 8 * kg)
                      : *reinterpret_cast<const uint4*>(
                            R + m * kDR + 8 * ((4 * (s - kLSteps) + kg) ^ (m & 7)));
        }
      };
      constexpr int kQA = 4;  // A-operand buffers: reads run three k-steps ahead
      uint4 ca[kQA][2];
#pragma unroll
      for (int i = 0; i < kQA - 1; ++i) read_a(i, ca[i]);
#pragma unroll
      for (int s = 0; s < kQSteps; ++s) {
        if (s + kQA - 1 < kQSteps) read_a(s + kQA - 1, ca[(s + kQA - 1) % kQA]);
#pragma unroll
        for (int t = 0; t < 2; ++t) {
#pragma unroll
          for (int ht = 0; ht < HT; ++ht) {
            sacc[ht][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, ca[s % kQA][t]), __builtin_bit_cast(bf16x8, qh[ht][s]),
                sacc[ht][t], 0, 0, 0);
            if (s < kLSteps)
              sacc[ht][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                  __builtin_bit_cast(bf16x8, ca[s % kQA][t]),
                  __builtin_bit_cast(bf16x8, ql[ht][s]), sacc[ht][t], 0, 0, 0);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }

      // Online softmax per head (log2 units) with a lazy reference: the
      // weights are 2^(s - m_ref); m_ref moves (and the accumulators are
      // rescaled) only when a chunk's maximum passes it by more than
      // kLazy, so weights stay below 2^kLazy and the accumulators are not
      // touched by the vector ALU on most chunks.
      float sv[HT][8];
      bool grow = false;
#pragma unroll
      for (int ht = 0; ht < HT; ++ht) {
        float mx = -INFINITY;
#pragma unroll
        for (int t = 0; t < 2; ++t)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const bool valid = c + 16 * t + 4 * kg + i < n_tok;
            sv[ht][4 * t + i] = valid ? sacc[ht][t][i] * a.scale_log2 : -INFINITY;
            mx = fmaxf(mx, sv[ht][4 * t + i]);
          }
        mx = xg_max(mx);
        grow |= mx > m_run[ht] + kLazy;
        sacc[ht][0][0] = mx;  // reuse: the chunk maximum of this lane's head
      }
      if (__builtin_amdgcn_ballot_w64(grow) != 0) {  // rare after the first chunk
#pragma unroll
        for (int ht = 0; ht < HT; ++ht) {
          const float mx = sacc[ht][0][0];
          if (mx > m_run[ht] + kLazy) {
            const float alpha = exp2f(m_run[ht] - mx);  // 0 on the first chunk
            l_run[ht] *= alpha;
            m_run[ht] = mx;
#pragma unroll
            for (int db = 0; db < kVBlocks; ++db) acc[ht][db] *= alpha;
          }
        }
      }
      uint4 phi[HT], plo[HT];
#pragma unroll
      for (int ht = 0; ht < HT; ++ht) {
        float ls = 0.f;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          // v_exp_f32 itself: results below 2^-126 flush to zero, which a
          // softmax weight can afford (exp2f adds a denormal-range fix-up,
          // four more instructions per weight)
          sv[ht][j] = __builtin_amdgcn_exp2f(sv[ht][j] - m_run[ht]);
          ls += sv[ht][j];
        }
        l_run[ht] += ls;
        // k-slots 8kg..8kg+7 of the 32-token block are tokens 4kg..4kg+3 of
        // the first tile and of the second: exactly the S^T entries held here.
        split8_trunc(sv[ht], phi[ht], plo[ht]);
      }

      // O^T += C^T P^T: the latent columns read transposed from LDS in the
      // same token order as the P slots.
      const uint16_t* r0 = C + (4 * kg + (r16 >> 2)) * kLPitch + 4 * (r16 & 3);
      const uint16_t* r1 = r0 + 16 * kLPitch;
      constexpr int kVA = 6;  // reads run five dim blocks ahead
      bf16x8 vA[kVA];
      auto read_v = [&](int db) {
        const bf16x4 va = lds_read_tr(r0 + 16 * db);
        const bf16x4 vb = lds_read_tr(r1 + 16 * db);
        return __builtin_shufflevector(va, vb, 0, 1, 2, 3, 4, 5, 6, 7);
      };
#pragma unroll
      for (int i = 0; i < kVA - 1; ++i) vA[i] = read_v(i);
#pragma unroll
      for (int db = 0; db < kVBlocks; ++db) {
        if (db + kVA - 1 < kVBlocks) vA[(db + kVA - 1) % kVA] = read_v(db + kVA - 1);
#pragma unroll
        for (int ht = 0; ht < HT; ++ht) {
          acc[ht][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              vA[db % kVA], __builtin_bit_cast(bf16x8, phi[ht]), acc[ht][db], 0, 0, 0);
          acc[ht][db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              vA[db % kVA], __builtin_bit_cast(bf16x8, plo[ht]), acc[ht][db], 0, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    // the padding chunks requested past the end land before the stages are
    // reused
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));

    // Partial results of this unit: (max, sum) per head and the unnormalised
    // latent accumulator.
#pragma unroll
    for (int ht = 0; ht < HT; ++ht) {
      const float l = xg_sum(l_run[ht]);
      const int head = head0 + 16 * ht + r16;
      const size_t prow = ((size_t)lb * a.n_split + split) * a.H + head;
      float* dst = a.part_acc + prow * kDC + 4 * kg;
#pragma unroll
      for (int db = 0; db < kVBlocks; ++db)
        *reinterpret_cast<float4*>(dst + 16 * db) =
            make_float4(acc[ht][db][0], acc[ht][db][1], acc[ht][db][2], acc[ht][db][3]);
      if (kg == 0) {
        a.part_ml[prow * 2] = m_run[ht];
        a.part_ml[prow * 2 + 1] = l;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// 3. merge the splits, o = W_UV[h] o~, lse
// ---------------------------------------------------------------------------
constexpr int kOPitch = kDC + 8;  // LDS pitch of the o~ tiles (elements)

__global__ __launch_bounds__(kMThreads, 2) void mla_out_kernel(MlaArgs a) {
  __shared__ __align__(16) uint16_t ohi[16 * kOPitch];
  __shared__ __align__(16) uint16_t olo[16 * kOPitch];
  __shared__ float wsp[16][17];  // per sequence: split weights, then the lse
  __shared__ float2 wml[kMMaxSplitCount][16];  // per split and sequence: (max, sum)

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int r16 = lane & 15;
  const int kg = lane >> 4;
  const int layer = blockIdx.x / a.H;
  const int h = blockIdx.x - layer * a.H;
  const uint16_t* w = a.w_uv + ((size_t)layer * a.H + h) * kDVo * kDC;

  // this wavefront's rows of W_UV[h] (v-tiles 2w, 2w+1), requested first so
  // that they stream in while the latent outputs are merged
  uint4 wr[2][kDC / 32];
#pragma unroll
  for (int vt = 0; vt < 2; ++vt) {
    const uint16_t* wp = w + (size_t)(32 * wave + 16 * vt + r16) * kDC + 8 * kg;
#pragma unroll
    for (int s = 0; s < kDC / 32; ++s) wr[vt][s] = ldg16_stream(wp + 32 * s);
  }
  constexpr int kItems = 16 * (kDC / 8) / kMThreads;  // (sequence, 8 dims) items per thread
  for (int b0 = 0; b0 < a.B; b0 += 16) {
    // Everything the merge reads is requested before the first wait: the
    // first split's partials of this thread's items and one (sequence, split)
    // pair of (max, sum) per thread.  (Loads retire in order, so a chain of
    // dependent loads here would queue each link behind the W_UV rows.)
    float4 x0[kItems][2];
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
      const int e = tid + i * kMThreads;
      const int t = e / (kDC / 8), c8 = e - t * (kDC / 8);
      const int b = min(b0 + t, a.B - 1);
      const float* src =
          a.part_acc + (((size_t)layer * a.B + b) * a.n_split * a.H + h) * kDC + 8 * c8;
      x0[i][0] = *reinterpret_cast<const float4*>(src);
      x0[i][1] = *reinterpret_cast<const float4*>(src + 4);
    }
    static_assert(kMMaxSplitCount * 16 == kMThreads, "one (split, sequence) pair per thread");
    const int ms_s = tid >> 4;
    const int ms_b = min(b0 + (tid & 15), a.B - 1);
    float2 ml = make_float2(-INFINITY, 0.f);
    if (ms_s < a.n_split)
      ml = *reinterpret_cast<const float2*>(
          a.part_ml + ((((size_t)layer * a.B + ms_b) * a.n_split + ms_s) * a.H + h) * 2);
    __syncthreads();  // the previous group's o~ tiles and weights are no longer read
    wml[ms_s][tid & 15] = ml;
    __syncthreads();
    // split weights w_s = 2^(m_s - M) / sum_s' 2^(m_s' - M) l_s' per sequence
    if (tid < 16 && b0 + tid < a.B) {
      float M = -INFINITY;
      for (int s = 0; s < a.n_split; ++s) M = fmaxf(M, wml[s][tid].x);
      float L = 0.f;
      for (int s = 0; s < a.n_split; ++s)
        L += M == -INFINITY ? 0.f : exp2f(wml[s][tid].x - M) * wml[s][tid].y;
      const float inv = L > 0.f ? 1.f / L : 0.f;
      for (int s = 0; s < a.n_split; ++s) {
        const float ms = wml[s][tid].x;
        wsp[tid][s] = (L > 0.f && ms != -INFINITY) ? exp2f(ms - M) * inv : 0.f;
      }
      wsp[tid][16] = L > 0.f ? (M + log2f(L)) * kLn2 : -INFINITY;
    }
    __syncthreads();
    // o~ of sequences b0 .. b0+15 as bf16 high + low parts (zero past B)
#pragma unroll
    for (int i = 0; i < kItems; ++i) {
      const int e = tid + i * kMThreads;
      const int t = e / (kDC / 8), c8 = e - t * (kDC / 8);
      const int b = b0 + t;
      float v[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) v[j] = 0.f;
      if (b < a.B) {
        const size_t base = ((size_t)layer * a.B + b) * a.n_split;
        for (int s = 0; s < a.n_split; ++s) {
          const float ws = wsp[t][s];
          float4 y0 = x0[i][0], y1 = x0[i][1];
          if (s > 0) {
            const float* src = a.part_acc + ((base + s) * a.H + h) * kDC + 8 * c8;
            y0 = *reinterpret_cast<const float4*>(src);
            y1 = *reinterpret_cast<const float4*>(src + 4);
          }
          v[0] += ws * y0.x; v[1] += ws * y0.y; v[2] += ws * y0.z; v[3] += ws * y0.w;
          v[4] += ws * y1.x; v[5] += ws * y1.y; v[6] += ws * y1.z; v[7] += ws * y1.w;
        }
      }
      uint4 hi, lo;
      split8(v, hi, lo);
      *reinterpret_cast<uint4*>(ohi + t * kOPitch + 8 * c8) = hi;
      *reinterpret_cast<uint4*>(olo + t * kOPitch + 8 * c8) = lo;
    }
    __syncthreads();

    // out^T[v][b] = W_UV[h][v][:] . o~[b][:]: wavefront w owns v-tiles 2w, 2w+1.
    floatx4 acc[2];
#pragma unroll
    for (int vt = 0; vt < 2; ++vt) acc[vt] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < kDC / 32; ++s) {
      const uint4 bh = *reinterpret_cast<const uint4*>(ohi + r16 * kOPitch + 32 * s + 8 * kg);
      const uint4 bl = *reinterpret_cast<const uint4*>(olo + r16 * kOPitch + 32 * s + 8 * kg);
#pragma unroll
      for (int vt = 0; vt < 2; ++vt) {
        acc[vt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8, wr[vt][s]), __builtin_bit_cast(bf16x8, bh), acc[vt], 0, 0, 0);
        acc[vt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
            __builtin_bit_cast(bf16x8, wr[vt][s]), __builtin_bit_cast(bf16x8, bl), acc[vt], 0, 0, 0);
      }
    }
    // lane (b = r16, kg) holds out[b][v = 32w + 16vt + 4kg + i]
    const int b = b0 + r16;
    if (b < a.B) {
      float* dst = a.out + (((size_t)layer * a.B + b) * a.H + h) * kDVo + 32 * wave + 4 * kg;
#pragma unroll
      for (int vt = 0; vt < 2; ++vt)
        *reinterpret_cast<float4*>(dst + 16 * vt) =
            make_float4(acc[vt][0], acc[vt][1], acc[vt][2], acc[vt][3]);
      if (a.lse && wave == 0 && kg == 0)
        a.lse[((size_t)layer * a.B + b) * a.H + h] = wsp[r16][16];
    }
  }
}

// Splits of the selection: enough work units for 256 CUs (a fixed target,
// so that the workspace size does not depend on the device), 256..2048
// tokens per unit, at most 16 units per (layer, sequence).
struct MlaPlan {
  int n_split, split_tokens, n_units, n_hg, n_items;
};

MlaPlan mla_plan(const MlaDims& d) {
  constexpr int kTargetUnits = 256;
  const int groups = d.n_layers * d.B * (d.H / 64);
  MlaPlan p;
  const int want = groups >= kTargetUnits ? 1 : (kTargetUnits + groups - 1) / groups;
  int split = (d.k_max + want - 1) / want;
  const int at_most_16 = (d.k_max + kMMaxSplitCount - 1) / kMMaxSplitCount;
  split = split < at_most_16 ? at_most_16 : split;
  split = (split + kMChunk - 1) / kMChunk * kMChunk;
  split = split < kMMinSplit ? kMMinSplit : split;
  split = split > kMMaxSplit ? kMMaxSplit : split;
  p.split_tokens = split;
  p.n_split = (d.k_max + split - 1) / split;
  p.n_hg = d.H / 64;
  p.n_units = d.n_layers * d.B * p.n_split;
  p.n_items = (p.n_units + 7) / 8 * 8 * p.n_hg;
  return p;
}

size_t qt_bytes(const MlaDims& d) {
  return align_up(sizeof(uint16_t) * (size_t)d.n_layers * d.B * d.H * kQT);
}
size_t part_acc_bytes(const MlaDims& d, int n_split) {
  return align_up(sizeof(float) * (size_t)d.n_layers * d.B * n_split * d.H * kDC);
}

}  // namespace

size_t mla_ws_bytes(const MlaDims& d) {
  const int ns = mla_plan(d).n_split;
  return qt_bytes(d) + part_acc_bytes(d, ns) +
         align_up(sizeof(float) * (size_t)d.n_layers * d.B * ns * d.H * 2);
}

hipError_t launch_mla(const MlaDims& d, const uint16_t* q, const uint16_t* ckv,
                      const uint16_t* w_uk, const uint16_t* w_uv, const int32_t* idx,
                      const int32_t* counts, float* out, float* lse, void* ws, hipStream_t s) {
  const MlaPlan p = mla_plan(d);
  const int n_cu = device_cu_count();
  MlaArgs a;
  a.q = q;
  a.ckv = ckv;
  a.w_uk = w_uk;
  a.w_uv = w_uv;
  a.idx = idx;
  a.counts = counts;
  char* base = static_cast<char*>(ws);
  a.qt = reinterpret_cast<uint16_t*>(base);
  base += qt_bytes(d);
  a.part_acc = reinterpret_cast<float*>(base);
  base += part_acc_bytes(d, p.n_split);
  a.part_ml = reinterpret_cast<float*>(base);
  a.out = out;
  a.lse = lse;
  a.stride_layer = d.stride_layer;
  a.stride_b = d.stride_b;
  a.B = d.B;
  a.H = d.H;
  a.k_max = d.k_max;
  a.L_cap = d.L_cap;
  a.n_layers = d.n_layers;
  a.n_split = p.n_split;
  a.split_tokens = p.split_tokens;
  a.n_units = p.n_units;
  a.n_hg = p.n_hg;
  a.n_items = p.n_items;
  a.scale_log2 = d.scale * kLog2e;

  const int grid_lh = d.n_layers * d.H;
  // a multiple of 16 keeps the two head groups of a unit on one XCD
  const int grid = p.n_items < n_cu ? p.n_items : (n_cu / 16 > 0 ? n_cu / 16 * 16 : n_cu);
  const dim3 abs_block(64);
  if (d.B == 1)
    hipLaunchKernelGGL((mla_absorb_kernel<1>), dim3(grid_lh), abs_block, 0, s, a);
  else if (d.B <= 4)
    hipLaunchKernelGGL((mla_absorb_kernel<4>), dim3(grid_lh), abs_block, 0, s, a);
  else
    hipLaunchKernelGGL((mla_absorb_kernel<8>), dim3(grid_lh), abs_block, 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((mla_attn_kernel<1>), dim3(grid), dim3(kMThreads), 0, s, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(mla_out_kernel, dim3(grid_lh), dim3(kMThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace spec
