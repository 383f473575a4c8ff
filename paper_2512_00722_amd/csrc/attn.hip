// Sparse GQA decode attention on gfx950 (SpeContext Eq. 1 over the selected
// tokens; Sec. 4.3 "Support for GQA": the G query heads of a group share one
// KV head, which is read directly -- no repeat_kv copy).
//
// Flash decode over work units (layer, sequence, KV head g, split of the
// selection).  One workgroup per CU runs one wavefront per SIMD; its
// wavefronts take units from a contiguous range on demand.  A wavefront walks
// its unit in chunks of 32 selected tokens:
//  * the unit's row indices are staged in LDS first, so no chunk waits on an
//    index load;
//  * S^T = K Q^T on the matrix cores (v_mfma_f32_16x16x32_bf16): A = 16
//    selected K rows, each lane feeding one 16-byte slice of one row straight
//    from HBM (no LDS staging, no conversion); B = Q^T with the G query heads
//    of the group as columns (columns >= G are zero).  Only G/16 of the tile
//    is useful, which does not matter: the op is HBM-bound;
//  * online softmax in log2 units (scale and log2(e) folded into one
//    multiply); the four lanes that hold one head combine with permlane swaps;
//  * O^T += V^T P^T on the matrix cores: V rows arrive as 16-byte loads (four
//    whole 256-byte rows per instruction), are staged in LDS and read back
//    transposed with ds_read_b64_tr_b16; P is split into a bf16 high part and
//    a bf16 low part (two MFMAs), which keeps it to ~2^-16 relative;
//  * K and V of chunk c+1 are requested as soon as chunk c's registers are
//    consumed and stay in flight through chunk c's softmax and MFMAs;
//  * when a wavefront has several units they are pipelined: when it starts a
//    unit it also takes its next one and requests that unit's count, row indices and queries
//    together (the indices unconditionally; the count only masks them), and
//    stages its rows in the other half of a double-buffered row area.  The
//    last chunk's refill then requests the next unit's first chunk, so a unit
//    boundary costs no round trip.
// The workgroups own contiguous ranges of a permuted unit order (groups of a
// (layer, sequence, split) spread over the whole range), so that ragged
// selections even out across workgroups.  Pipelined launches over batches
// of unequal selections deal the groups to the workgroups by selection size
// instead (longest first, in a snake), which evens them out further.
// A unit that covers a whole selection normalises and writes out/lse itself;
// split selections leave (max, sum, acc) partials that a second kernel merges
// with a log-sum-exp combine.
#include <stdlib.h>
#include <string.h>

#include "device_common.h"
#include "internal.h"

namespace spec {
namespace {

#ifndef SPEC_ATTN_CHUNK
#define SPEC_ATTN_CHUNK 32
#endif
#ifndef SPEC_ATTN_NT
#define SPEC_ATTN_NT 1
#endif
#ifndef SPEC_ATTN_WPE
#define SPEC_ATTN_WPE 2  // wavefronts per SIMD the register budget is sized for
#endif
#ifndef SPEC_ATTN_WAVES
#define SPEC_ATTN_WAVES 4
#endif
constexpr int kWaves = SPEC_ATTN_WAVES;   // wavefronts per workgroup
constexpr int kChunk = SPEC_ATTN_CHUNK;   // selected tokens per inner step (32 or 64)
constexpr int kTiles = kChunk / 16;       // 16-token MFMA tiles per chunk
constexpr int kVRows = kChunk / 4;        // V rows per lane per chunk
constexpr int kD = 128;                   // head dimension
constexpr int kMaxSplit = 2048;           // longest split (tokens per work item)
#ifndef SPEC_ATTN_MIN_SPLIT
#define SPEC_ATTN_MIN_SPLIT 256
#endif

constexpr int kMinSplitTokens = SPEC_ATTN_MIN_SPLIT;
#ifndef SPEC_ATTN_SLOT_UNITS
#define SPEC_ATTN_SLOT_UNITS 1
#endif
// Work units per resident wavefront the selections are split into when there
// are fewer (layer, sequence, KV head) groups than wavefronts.
constexpr int kSlotUnits = SPEC_ATTN_SLOT_UNITS;

// K/V rows are read once per launch: stream them past the caches.
__device__ __forceinline__ uint4 ldkv(const uint16_t* p) {
#if SPEC_ATTN_NT
  return ldg16_stream(p);
#else
  return ldg16(p);
#endif
}

// How the selection of a (layer, sequence, KV head) group is covered:
//  kDirect:         one work unit per group; the wave writes out/lse.
//  kGlobalPartials: the selection is split over several units; partial
//                   results go to the workspace and a second kernel merges
//                   them.
enum AttnMode { kDirect = 0, kGlobalPartials = 1 };

// Where a unit's K/V rows come from:
//  kKvIndexed: the cache, at the selected token indices (idx);
//  kKvCompact: the compact slot buffers, slots 0 .. count-1;
//  kKvElastic: the slot buffers, except the slots an elastic update has just
//              assigned (src[b][slot] = token >= 0): those rows are read from
//              the cache and written into their slot as they stream through
//              (Sec. 5.4's loads fused into the attention's reads).
enum KvMode { kKvIndexed = 0, kKvCompact = 1, kKvElastic = 2 };

struct AttnArgs {
  const uint16_t* q;      // [n_layers][B][H_q][d]
  const uint16_t* k;      // indexed, elastic: cache; compact: [n_layers][B][k_max][H_kv][d]
  const uint16_t* v;
  const int32_t* idx;     // [B][k_max] (indexed mode)
  uint16_t* kbuf;         // elastic: slot buffers [n_layers][B][k_max][H_kv][d]
  uint16_t* vbuf;
  const int32_t* src;     // elastic: [B][k_max] token loaded into the slot, or -1
  const int32_t* fused;   // elastic: [B] or null; 0: the sequence's rows are all in the slots
  const int32_t* counts;  // [B]
  float* part_acc;        // [n_layers*B][n_split][H_q][d]
  float* part_ml;         // [n_layers*B][n_split][H_q][2]
  float* out;             // [n_layers*B][H_q][d]
  float* lse;             // [n_layers*B][H_q] or null
  int64_t stride_layer;   // elements between layers of the cache (indexed, elastic)
  int64_t stride_b;       // elements between sequences of the cache
  int B, H_q, H_kv, G, k_max, L_cap, n_split, split_tokens, n_items;
  int R;                  // column groups per KV head (1; G/16 for more than 16 query heads)
                          // G above: query heads per column group (at most 16)
  int mode;               // kDirect or kGlobalPartials
  int n_groups, perm;     // work order: group g (G_u = H_kv R consecutive units) runs as group
                          // (g perm) mod n_groups, perm coprime to n_groups
  int n_sets;             // 1: idx [B][k_max]; H_kv: idx [B][H_kv][k_max], one set per KV head
  float scale_log2;       // scale * log2(e)
  int sorted;             // pipelined launches: groups by selection size (see attn_split_kernel)
};

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// LDS row pitch of a staged V tile in bf16: 288 bytes, so that the rows of
// one transpose read start 32 bytes apart and spread over the banks.
constexpr int kVPitch = kD + 16;

__device__ __forceinline__ uint32_t f2bf_rne(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
}

// 8 probabilities -> bf16 hi part and bf16 lo part (p - hi), packed for MFMA.
__device__ __forceinline__ void split_bf16x8(const float* p, bf16x8& hi, bf16x8& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const uint32_t h0 = f2bf_rne(p[2 * j]), h1 = f2bf_rne(p[2 * j + 1]);
    const uint32_t l0 = f2bf_rne(p[2 * j] - __uint_as_float(h0 << 16));
    const uint32_t l1 = f2bf_rne(p[2 * j + 1] - __uint_as_float(h1 << 16));
    h[j] = h0 | (h1 << 16);
    l[j] = l0 | (l1 << 16);
  }
  hi = __builtin_bit_cast(bf16x8, make_uint4(h[0], h[1], h[2], h[3]));
  lo = __builtin_bit_cast(bf16x8, make_uint4(l[0], l[1], l[2], l[3]));
}

// max / sum over the four lanes {l, l^16, l^32, l^48} (one head's lanes).
__device__ __forceinline__ float xgroup_max(float v) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float xgroup_sum(float v) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  v = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

// Transposing LDS read: within each 16-lane group, lane i receives element
// (i & 3) of the 8-byte chunks read by lanes (i >> 2) + 4j, j = 0..3.
__device__ __forceinline__ bf16x4 lds_read_tr(const uint16_t* p) {
  return __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
      (__attribute__((address_space(3))) bf16x4*)(p));
}

// Rows staged per unit: up to kMaxSplit rows of the selection split plus one
// chunk of padding (the software pipeline reads one chunk past the end when
// no unit follows).
constexpr int kRowsCap = kMaxSplit + kChunk;
constexpr int kRowLoads = kMaxSplit / 64;  // index loads per lane for one unit
// Sequences a launch may rank by selection size (one per thread of the workgroup).
constexpr int kSortMaxB = kWaves * 64;

// One work unit: (layer, sequence, KV-head column group, split).  A group of
// more than 16 query heads is covered by R column groups of 16 (gv = g R ..
// g R + R - 1), each a unit of its own that reads KV head g; the query heads
// of column group gv are gv G .. gv G + G - 1.
struct Unit {
  int lb, b, gv, g, split, j0;
  int n_tok;  // tokens of the unit (<= 0: none), known once the count has arrived
};

__device__ __forceinline__ Unit decode_unit(const AttnArgs& a, int item) {
  Unit u;
  u.gv = item % (a.H_kv * a.R);
  u.g = u.gv / a.R;
  const int rest = item / (a.H_kv * a.R);
  u.split = rest % a.n_split;
  u.lb = rest / a.n_split;  // layer * B + b
  u.b = u.lb % a.B;
  u.j0 = u.split * a.split_tokens;
  u.n_tok = 0;
  return u;
}

// Elastic mode: the staged value of a row is the cache token to read (and
// write into the slot), or -1 - slot for a row read from its slot.  Other
// modes stage the token or slot index clamped into range.
template <int KV>
__device__ __forceinline__ int elastic_row(int v, int slot, int L_cap) {
  if (KV != kKvElastic) return clampi(v, 0, L_cap - 1);
  return v >= 0 ? min(v, L_cap - 1) : -1 - slot;
}
template <int KV>
__device__ __forceinline__ const uint16_t* row_ptr(const uint16_t* base, const uint16_t* buf,
                                                   int r, int64_t rs) {
  if (KV != kKvElastic) return base + (int64_t)r * rs;
  return r >= 0 ? base + (int64_t)r * rs : buf + (int64_t)(-1 - r) * rs;
}

// The rows of one chunk that came from the cache, written into their slots
// (dst: the chunk's first slot, this KV head): the data registers as loaded,
// so each slot receives the cache row bit for bit.  n: tokens of the unit
// from this chunk on.
__device__ __forceinline__ void store_k_rows(const int* rc, const uint4 (&kr)[kTiles][4],
                                             uint16_t* dst, int64_t rs, int n, int kg, int r16) {
#pragma unroll
  for (int t = 0; t < kTiles; ++t) {
    const int j = 16 * t + r16;
    if (rc[j] >= 0 && j < n) {
      uint16_t* p = dst + (int64_t)j * rs + 8 * kg;
#pragma unroll
      for (int s = 0; s < 4; ++s) *reinterpret_cast<uint4*>(p + 32 * s) = kr[t][s];
    }
  }
}
__device__ __forceinline__ void store_v_rows(const int* rc, const uint4 (&vr)[kVRows],
                                             uint16_t* dst, int64_t rs, int n, int kg, int r16) {
#pragma unroll
  for (int r = 0; r < kVRows; ++r) {
    const int j = 4 * r + kg;
    if (rc[j] >= 0 && j < n) *reinterpret_cast<uint4*>(dst + (int64_t)j * rs + 8 * r16) = vr[r];
  }
}

// One unit from a cold start (a wavefront with a single unit): count, then
// indices staged in LDS, then the first chunk.
template <int KV>
__device__ __forceinline__ void process_item(const AttnArgs& a, const int item, const int lane,
                                             uint16_t* V, int* rows) {
  // A group of more than 16 query heads is covered by R column groups of
  // 16 (gv = g R .. g R + R - 1), each a unit of its own that reads KV head
  // g; the query heads of column group gv are gv G .. gv G + G - 1.
  const int G = a.G;
  const int gv = item % (a.H_kv * a.R);
  const int g = gv / a.R;
  const int rest = item / (a.H_kv * a.R);
  const int split = rest % a.n_split;
  const int lb = rest / a.n_split;  // layer * B + b
  const int b = lb % a.B;
  const int layer = lb / a.B;
  const int count = __builtin_amdgcn_readfirstlane(clampi(a.counts[b], 0, a.k_max));
  const int j0 = split * a.split_tokens;
  const int r16e = lane & 15;
  if (j0 >= count) {  // uniform per wavefront
    if (a.mode == kDirect && r16e < G) {  // no tokens: out = 0, lse = -inf
      const size_t orow = (size_t)lb * a.H_q + (size_t)gv * G + r16e;
      float* dst = a.out + orow * kD + 4 * (lane >> 4);
#pragma unroll
      for (int db = 0; db < 8; ++db)
        *reinterpret_cast<float4*>(dst + 16 * db) = make_float4(0.f, 0.f, 0.f, 0.f);
      if (a.lse && (lane >> 4) == 0) a.lse[orow] = -INFINITY;
    }
    return;
  }
  const int n_tok = min(a.split_tokens, count - j0);  // tokens of this work item

  const int64_t rs = (int64_t)a.H_kv * kD;  // elements per token row
  // kb/vb: the rows a staged row value r >= 0 addresses (the cache, or the
  // slot buffers in compact mode); kbf/vbf: elastic mode's slot buffers, for
  // r < 0 (slot -1 - r).
  const int64_t coff = (int64_t)layer * a.stride_layer + (int64_t)b * a.stride_b + g * kD;
  const int64_t boff = (int64_t)lb * a.k_max * rs + g * kD;
  const uint16_t* kb = a.k + (KV == kKvCompact ? boff : coff);
  const uint16_t* vb = a.v + (KV == kKvCompact ? boff : coff);
  uint16_t* kbf = a.kbuf + boff;
  uint16_t* vbf = a.vbuf + boff;
  const bool writer = KV == kKvElastic && gv % a.R == 0;  // one column group writes the slots

  const int r16 = lane & 15;  // head of this lane (MFMA column); token of a K tile row
  const int kg = lane >> 4;   // MFMA k-group; also the token phase of V loads
  // B operand of S^T = K Q^T: Q^T column r16 = query head gv*G + r16 (zero if >= G),
  // dims 32s + 8kg .. +8.  Loaded together with the row indices.
  bf16x8 qf[4];
  {
    const uint16_t* qp = a.q + ((size_t)lb * a.H_q + gv * G + (r16 < G ? r16 : 0)) * kD + 8 * kg;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      uint4 w = r16 < G ? ldg16(qp + 32 * s) : make_uint4(0, 0, 0, 0);
      qf[s] = __builtin_bit_cast(bf16x8, w);
    }
  }

  // Stage the rows of this item's tokens in LDS (masked tokens read row 0),
  // so that no chunk waits on an index load from memory.
  wave_sync_lds();  // the previous item's reads of rows/V are done
  {
    // All index loads are issued before any is used (one round trip), and
    // one chunk of padding follows the end: the software pipeline always
    // prefetches the next chunk, and padding rows all read row 0 (cache hits).
    const int32_t* idx_b =
        KV == kKvIndexed ? a.idx + ((size_t)b * a.n_sets + (a.n_sets > 1 ? g : 0)) * a.k_max + j0
        : KV == kKvElastic ? a.src + (size_t)b * a.k_max + j0
                           : nullptr;
    const bool fz = KV == kKvElastic && (a.fused == nullptr || a.fused[b] != 0);
    const int n_pad = (n_tok + kChunk - 1) / kChunk * kChunk + kChunk;
    constexpr int kColdRowLoads = (kMaxSplit + kChunk + 63) / 64;
    int rv[kColdRowLoads];
#pragma unroll
    for (int m = 0; m < kColdRowLoads; ++m) {
      const int j = lane + 64 * m;
      rv[m] = KV == kKvElastic ? -1 : 0;  // padding: the unit's first slot, or row 0
      if (j < n_tok && (KV != kKvElastic || fz)) rv[m] = KV == kKvCompact ? j0 + j : idx_b[j];
    }
#pragma unroll
    for (int m = 0; m < kColdRowLoads; ++m) {
      const int j = lane + 64 * m;
      if (j < n_pad)
        rows[j] = elastic_row<KV>(rv[m], j < n_tok ? j0 + j : j0, a.L_cap);
    }
  }

  wave_sync_lds();

  // K rows in the MFMA A-operand layout: tile t, token 16t + r16, dims
  // 32s + 8kg .. +8.  V rows: load r brings token 4r + kg, dims 8 r16 .. +8,
  // i.e. four whole 256-byte rows per instruction.
  auto load_k = [&](int c, uint4 (&kr)[kTiles][4]) {
    const int* rc = rows + c;
#pragma unroll
    for (int t = 0; t < kTiles; ++t) {
      const uint16_t* p = row_ptr<KV>(kb, kbf, rc[16 * t + r16], rs) + 8 * kg;
#pragma unroll
      for (int s = 0; s < 4; ++s) kr[t][s] = ldkv(p + 32 * s);
    }
  };
  auto load_v = [&](int c, uint4 (&vr)[kVRows]) {
    const int* rc = rows + c;
#pragma unroll
    for (int r = 0; r < kVRows; ++r)
      vr[r] = ldkv(row_ptr<KV>(vb, vbf, rc[4 * r + kg], rs) + 8 * r16);
  };

  float m_run = -INFINITY, l_run = 0.f;  // head r16
  floatx4 acc[8];                        // O^T[16db + 4kg + i][head r16]
#pragma unroll
  for (int db = 0; db < 8; ++db) acc[db] = floatx4{0.f, 0.f, 0.f, 0.f};

  // Single register buffers, refilled as soon as they are consumed: V(c+1)
  // is requested right after V(c) is staged in LDS, K(c+1) right after the
  // Q.K^T MFMAs have read K(c); both stay in flight through the softmax and
  // the P.V MFMAs of chunk c.  Loads retire in issue order, so each wait is
  // a partial one.  The prefetch past the last chunk reads padding rows
  // (row 0, cache hits).
  uint4 kraw[kTiles][4], vraw[kVRows];
  load_v(0, vraw);
  __builtin_amdgcn_sched_barrier(0);
  load_k(0, kraw);
  __builtin_amdgcn_sched_barrier(0);
  for (int c = 0; c < n_tok; c += kChunk) {
#pragma unroll
    for (int r = 0; r < kVRows; ++r)
      *reinterpret_cast<uint4*>(V + (4 * r + kg) * kVPitch + 8 * r16) = vraw[r];
    if (writer) store_v_rows(rows + c, vraw, vbf + (int64_t)(j0 + c) * rs, rs, n_tok - c, kg, r16);
    load_v(c + kChunk, vraw);
    __builtin_amdgcn_sched_barrier(0);  // keep the refill here: issue order = retire order

    // S^T tiles: lane holds S[head r16][token 16t + 4kg + i].
    floatx4 sacc[kTiles];
#pragma unroll
    for (int t = 0; t < kTiles; ++t) {
      sacc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < 4; ++s)
        sacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kraw[t][s]),
                                                          qf[s], sacc[t], 0, 0, 0);
    }
    if (writer) store_k_rows(rows + c, kraw, kbf + (int64_t)(j0 + c) * rs, rs, n_tok - c, kg, r16);
    load_k(c + kChunk, kraw);
    __builtin_amdgcn_sched_barrier(0);

    float sv[kTiles][4];
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < kTiles; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const bool valid = c + 16 * t + 4 * kg + i < n_tok;
        sv[t][i] = valid ? sacc[t][i] * a.scale_log2 : -INFINITY;
        mx = fmaxf(mx, sv[t][i]);
      }
    mx = xgroup_max(mx);
    const float mn = fmaxf(m_run, mx);
    const float alpha = exp2f(m_run - mn);
    float ls = 0.f;
#pragma unroll
    for (int t = 0; t < kTiles; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        sv[t][i] = exp2f(sv[t][i] - mn);
        ls += sv[t][i];
      }
    l_run = l_run * alpha + ls;
    m_run = mn;
#pragma unroll
    for (int db = 0; db < 8; ++db) acc[db] *= alpha;

    // O^T += V^T P^T on the matrix cores.  The k-slots 8kg..8kg+7 of a
    // 32-token block are tokens 4kg..4kg+3 of its first tile and of its
    // second tile: exactly the S^T entries this lane holds.
    wave_sync_lds();
#pragma unroll
    for (int kb2 = 0; kb2 < kChunk / 32; ++kb2) {
      float pv[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        pv[i] = sv[2 * kb2][i];
        pv[4 + i] = sv[2 * kb2 + 1][i];
      }
      bf16x8 phi, plo;
      split_bf16x8(pv, phi, plo);
      const uint16_t* r0 = V + (32 * kb2 + 4 * kg + (r16 >> 2)) * kVPitch + 4 * (r16 & 3);
      const uint16_t* r1 = r0 + 16 * kVPitch;
#pragma unroll
      for (int db = 0; db < 8; ++db) {
        const bf16x4 va = lds_read_tr(r0 + 16 * db);
        const bf16x4 vb4 = lds_read_tr(r1 + 16 * db);
        const bf16x8 vA = __builtin_shufflevector(va, vb4, 0, 1, 2, 3, 4, 5, 6, 7);
        acc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vA, phi, acc[db], 0, 0, 0);
        acc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vA, plo, acc[db], 0, 0, 0);
      }
    }
    wave_sync_lds();  // the V tile is rewritten by the next chunk
  }

  l_run = xgroup_sum(l_run);
  if (r16 < G) {
    if (a.mode == kDirect) {  // the whole selection: normalise and write the output
      const size_t orow = (size_t)lb * a.H_q + (size_t)gv * G + r16;
      const float inv = 1.f / l_run;
      float* dst = a.out + orow * kD + 4 * kg;
#pragma unroll
      for (int db = 0; db < 8; ++db)
        *reinterpret_cast<float4*>(dst + 16 * db) =
            make_float4(acc[db][0] * inv, acc[db][1] * inv, acc[db][2] * inv, acc[db][3] * inv);
      if (a.lse && kg == 0) a.lse[orow] = (m_run + log2f(l_run)) * kLn2;
    } else {
      const size_t prow = ((size_t)lb * a.n_split + split) * a.H_q + (size_t)gv * G + r16;
      float* dst = a.part_acc + prow * kD + 4 * kg;
#pragma unroll
      for (int db = 0; db < 8; ++db)
        *reinterpret_cast<float4*>(dst + 16 * db) =
            make_float4(acc[db][0], acc[db][1], acc[db][2], acc[db][3]);
      if (kg == 0) {
        a.part_ml[prow * 2] = m_run;
        a.part_ml[prow * 2 + 1] = l_run;
      }
    }
  }
}


// Dynamic LDS requested on top of the static arrays so that one workgroup
// takes more than half of a CU's 160 KiB: exactly one per CU.
constexpr size_t kLdsPerCU = 160 * 1024;
constexpr size_t static_lds(bool pipe) {
  return sizeof(uint16_t) * kWaves * kChunk * kVPitch + sizeof(int) * kWaves * (pipe ? 2 : 1) * kRowsCap +
         sizeof(int) * (pipe ? kSortMaxB : 1) + 16;
}
constexpr size_t lds_reserve(bool pipe) {
  return kLdsPerCU / 2 + 1024 > static_lds(pipe) ? kLdsPerCU / 2 + 1024 - static_lds(pipe) : 0;
}

// PIPE: some wavefront has more than one unit, and units are pipelined
// across their boundaries; otherwise each unit starts cold (the pipeline's
// bookkeeping made one-unit launches ~1.5 us slower).
template <int KV, bool PIPE>
__global__ __launch_bounds__(kWaves * 64) __attribute__((amdgpu_waves_per_eu(SPEC_ATTN_WPE)))
void attn_split_kernel(AttnArgs a) {
  __shared__ __align__(16) uint16_t vlds[kWaves][kChunk * kVPitch];
  __shared__ int rows_lds[kWaves][PIPE ? 2 : 1][kRowsCap];
  __shared__ int next_unit;
  __shared__ int seq_order[PIPE ? kSortMaxB : 1];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  // One workgroup per CU, one wavefront per SIMD.  Two wavefronts on a SIMD
  // do not progress at equal rates (the older one wins instruction issue), and
  // they add no bandwidth over one wavefront with its loads in flight, so the
  // CU runs one per SIMD.  The workgroup owns a contiguous range of the
  // permuted unit order; its wavefronts take them on demand from an LDS
  // counter, which evens out units of unequal length within the workgroup
  // (the permutation evens them out across workgroups).
  //
  // Sorted order (pipelined launches over ragged batches): the sequences are
  // ranked by selection size, longest first, and the (layer, sequence,
  // split) groups in that order are dealt to the workgroups in a snake
  // (row r of gridDim.x groups left to right for even r, right to left for
  // odd r), so that every workgroup receives about the same number of
  // tokens.  The units of one group (its KV heads) stay consecutive.
  // Selections of one size need no sorting: the permuted order is kept.
  bool sorted = false;
  if (PIPE && a.sorted) {
    int* cnt = &rows_lds[0][0][0];  // scratch until the first unit is staged
    const int t = threadIdx.x;      // kWaves * 64 = kSortMaxB >= B threads
    const int c = t < a.B ? clampi(a.counts[t], 0, a.k_max) : -1;
    cnt[t] = c;
    __syncthreads();
    sorted = !__syncthreads_and(t >= a.B || c == cnt[0]);  // uniform for the workgroup
    if (sorted && t < a.B) {
      int r = 0;
      for (int u = 0; u < a.B; ++u) {
        const int cu = cnt[u];
        r += cu > c || (cu == c && u < t);
      }
      seq_order[r] = t;
    }
  }
  const int per_block = (a.n_items + gridDim.x - 1) / gridDim.x;
  const int u0 = sorted ? 0 : blockIdx.x * per_block;
  const int u1 = min(u0 + per_block, a.n_items);
  if (threadIdx.x == 0) next_unit = u0;
  __syncthreads();
  auto take = [&]() -> int {
    int t = 0;
    if (lane == 0) t = atomicAdd(&next_unit, 1);
    const int unit = __builtin_amdgcn_readfirstlane(t);
    const int gu = a.H_kv * a.R;  // units per group (all column groups of one (layer, sequence, split))
    if (sorted) {
      const int row = unit / gu;
      const int col = (row & 1) ? (int)gridDim.x - 1 - (int)blockIdx.x : (int)blockIdx.x;
      const int64_t j = (int64_t)row * gridDim.x + col;  // group in size order
      if (j >= a.n_groups) return -1;  // uniform per wave; later rows are past the end too
      const int per_seq = a.n_groups / a.B;  // layers x splits
      const int rank = (int)(j / per_seq);
      const int rem = (int)(j - (int64_t)rank * per_seq);
      const int layer = rem / a.n_split;
      const int split = rem - layer * a.n_split;
      const int lb = layer * a.B + seq_order[rank];
      return (lb * a.n_split + split) * gu + (unit - row * gu);
    }
    if (unit >= u1) return -1;  // uniform per wave
    const int grp = unit / gu;
    return (int)(((int64_t)grp * a.perm) % a.n_groups) * gu + (unit - grp * gu);
  };

  if constexpr (!PIPE) {
    for (;;) {
      const int item = take();
      if (item < 0) return;  // uniform per wave: every wave ends here
      process_item<KV>(a, item, lane, vlds[wave], rows_lds[wave][0]);
    }
  } else {
  uint16_t* V = vlds[wave];
  const int r16 = lane & 15;  // head of this lane (MFMA column); token of a K tile row
  const int kg = lane >> 4;   // MFMA k-group; also the token phase of V loads
  const int64_t rs = (int64_t)a.H_kv * kD;  // elements per token row

  // The rows a staged value r >= 0 addresses (the cache; the slot buffers in
  // compact mode), and elastic mode's slot buffers (r < 0: slot -1 - r).
  auto kv_base = [&](const Unit& u, const uint16_t* p) -> const uint16_t* {
    if (KV != kKvCompact)
      return p + (int64_t)(u.lb / a.B) * a.stride_layer + (int64_t)u.b * a.stride_b + u.g * kD;
    return p + (int64_t)u.lb * a.k_max * rs + u.g * kD;
  };
  auto buf_base = [&](const Unit& u, uint16_t* p) -> uint16_t* {
    return KV == kKvElastic ? p + (int64_t)u.lb * a.k_max * rs + u.g * kD : nullptr;
  };

  // The loads that start a unit, all independent of each other: its count,
  // its row indices (all of a split's, clamped into the index row: the count
  // only masks them later) and its queries.  B operand of S^T = K Q^T: Q^T
  // column r16 = query head gv G + r16 (zero if >= G), dims 32s + 8kg .. +8.
  int cnt_raw, fz_raw = 1;
  int rv[kRowLoads];
  uint4 qraw[4];
  auto fetch = [&](const Unit& u) {
    cnt_raw = a.counts[u.b];
    if (KV == kKvElastic && a.fused) fz_raw = a.fused[u.b];
    const int32_t* idx_b =
        KV == kKvIndexed ? a.idx + ((size_t)u.b * a.n_sets + (a.n_sets > 1 ? u.g : 0)) * a.k_max
        : KV == kKvElastic ? a.src + (size_t)u.b * a.k_max
                           : nullptr;
    // loads past the split re-read its last index (one cache line)
    const int jmax = min(u.j0 + a.split_tokens, a.k_max) - 1;
#pragma unroll
    for (int m = 0; m < kRowLoads; ++m) {
      const int j = u.j0 + lane + 64 * m;
      rv[m] = KV == kKvCompact ? j : idx_b[min(j, jmax)];
    }
    const uint16_t* qp =
        a.q + ((size_t)u.lb * a.H_q + u.gv * a.G + (r16 < a.G ? r16 : 0)) * kD + 8 * kg;
#pragma unroll
    for (int s = 0; s < 4; ++s) qraw[s] = ldg16(qp + 32 * s);
  };
  // Rows of a unit's tokens into LDS: tokens past the unit, and the padding
  // chunk, read row 0 (elastic mode: the unit's first slot; cache hits).
  // Sets u.n_tok.
  auto stage = [&](Unit& u, int* rows) {
    const int count = __builtin_amdgcn_readfirstlane(clampi(cnt_raw, 0, a.k_max));
    u.n_tok = min(a.split_tokens, count - u.j0);
    const int pad = KV == kKvElastic ? -1 - u.j0 : 0;
    const bool fz = __builtin_amdgcn_readfirstlane(fz_raw) != 0;  // elastic: rows may come from the caches
#pragma unroll
    for (int m = 0; m < kRowLoads; ++m) {
      const int j = lane + 64 * m;
      rows[j] = j < u.n_tok ? elastic_row<KV>(fz ? rv[m] : -1, u.j0 + j, a.L_cap) : pad;
    }
    if (lane < kChunk) rows[kMaxSplit + lane] = pad;
  };

  // K rows in the MFMA A-operand layout: tile t, token 16t + r16, dims
  // 32s + 8kg .. +8.  V rows: load r brings token 4r + kg, dims 8 r16 .. +8,
  // i.e. four whole 256-byte rows per instruction.
  auto load_k = [&](const int* rc, const uint16_t* kb, const uint16_t* kbf,
                    uint4 (&kr)[kTiles][4]) {
#pragma unroll
    for (int t = 0; t < kTiles; ++t) {
      const uint16_t* p = row_ptr<KV>(kb, kbf, rc[16 * t + r16], rs) + 8 * kg;
#pragma unroll
      for (int s = 0; s < 4; ++s) kr[t][s] = ldkv(p + 32 * s);
    }
  };
  auto load_v = [&](const int* rc, const uint16_t* vb, const uint16_t* vbf, uint4 (&vr)[kVRows]) {
#pragma unroll
    for (int r = 0; r < kVRows; ++r)
      vr[r] = ldkv(row_ptr<KV>(vb, vbf, rc[4 * r + kg], rs) + 8 * r16);
  };

  int buf = 0;
  int item = take();
  if (item < 0) return;
  Unit cur = decode_unit(a, item);
  fetch(cur);
  wave_sync_lds();
  stage(cur, rows_lds[wave][buf]);
  wave_sync_lds();
  uint4 kraw[kTiles][4], vraw[kVRows];
  const uint16_t* kb = kv_base(cur, a.k);
  const uint16_t* vb = kv_base(cur, a.v);
  uint16_t* kbf = buf_base(cur, a.kbuf);
  uint16_t* vbf = buf_base(cur, a.vbuf);
  bf16x8 qf[4];
#pragma unroll
  for (int s = 0; s < 4; ++s)
    qf[s] = __builtin_bit_cast(bf16x8, r16 < a.G ? qraw[s] : make_uint4(0, 0, 0, 0));
  if (cur.n_tok > 0) {  // uniform per wavefront
    load_v(rows_lds[wave][buf], vb, vbf, vraw);
    __builtin_amdgcn_sched_barrier(0);
    load_k(rows_lds[wave][buf], kb, kbf, kraw);
    __builtin_amdgcn_sched_barrier(0);
  }

  for (;;) {
    // The next unit: its count, indices and queries are requested now and its
    // rows staged before this unit's chunks, so that this unit's last refill
    // can request the next unit's first chunk.
    const int nitem = take();
    Unit nxt = decode_unit(a, nitem < 0 ? 0 : nitem);
    bf16x8 qn[4];
    if (nitem >= 0) {
      fetch(nxt);
      wave_sync_lds();  // the previous unit's reads of this row buffer are done
      stage(nxt, rows_lds[wave][buf ^ 1]);
#pragma unroll
      for (int s = 0; s < 4; ++s)
        qn[s] = __builtin_bit_cast(bf16x8, r16 < a.G ? qraw[s] : make_uint4(0, 0, 0, 0));
    }
    // the next unit's chunk 0 is requested by this unit's last refill
    const bool chain = cur.n_tok > 0 && nitem >= 0 && nxt.n_tok > 0;
    const uint16_t* kbn = kv_base(nxt, a.k);
    const uint16_t* vbn = kv_base(nxt, a.v);
    uint16_t* kbfn = buf_base(nxt, a.kbuf);
    uint16_t* vbfn = buf_base(nxt, a.vbuf);
    const bool writer = KV == kKvElastic && cur.gv % a.R == 0;  // one column group writes
    const int* rows = rows_lds[wave][buf];
    const int* rows_n = rows_lds[wave][buf ^ 1];
    wave_sync_lds();

    const int n_tok = cur.n_tok;
    float m_run = -INFINITY, l_run = 0.f;  // head r16
    floatx4 acc[8];                        // O^T[16db + 4kg + i][head r16]
#pragma unroll
    for (int db = 0; db < 8; ++db) acc[db] = floatx4{0.f, 0.f, 0.f, 0.f};

    // Single register buffers, refilled as soon as they are consumed: V(c+1)
    // is requested right after V(c) is staged in LDS, K(c+1) right after the
    // Q.K^T MFMAs have read K(c); both stay in flight through the softmax and
    // the P.V MFMAs of chunk c.  Loads retire in issue order, so each wait is
    // a partial one.  After the last chunk the refill requests the next
    // unit's first chunk, or padding rows (row 0, cache hits) if none follows.
    for (int c = 0; c < n_tok; c += kChunk) {
      const bool last = c + kChunk >= n_tok;
      const int* rsrc = last && chain ? rows_n : rows + c + kChunk;
      const uint16_t* ksrc = last && chain ? kbn : kb;
      const uint16_t* vsrc = last && chain ? vbn : vb;
      const uint16_t* kfsrc = last && chain ? kbfn : kbf;
      const uint16_t* vfsrc = last && chain ? vbfn : vbf;
#pragma unroll
      for (int r = 0; r < kVRows; ++r)
        *reinterpret_cast<uint4*>(V + (4 * r + kg) * kVPitch + 8 * r16) = vraw[r];
      if (writer)
        store_v_rows(rows + c, vraw, vbf + (int64_t)(cur.j0 + c) * rs, rs, n_tok - c, kg, r16);
      load_v(rsrc, vsrc, vfsrc, vraw);
      __builtin_amdgcn_sched_barrier(0);  // keep the refill here: issue order = retire order

      // S^T tiles: lane holds S[head r16][token 16t + 4kg + i].
      floatx4 sacc[kTiles];
#pragma unroll
      for (int t = 0; t < kTiles; ++t) {
        sacc[t] = floatx4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < 4; ++s)
          sacc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kraw[t][s]),
                                                            qf[s], sacc[t], 0, 0, 0);
      }
      if (writer)
        store_k_rows(rows + c, kraw, kbf + (int64_t)(cur.j0 + c) * rs, rs, n_tok - c, kg, r16);
      load_k(rsrc, ksrc, kfsrc, kraw);
      __builtin_amdgcn_sched_barrier(0);

      float sv[kTiles][4];
      float mx = -INFINITY;
#pragma unroll
      for (int t = 0; t < kTiles; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const bool valid = c + 16 * t + 4 * kg + i < n_tok;
          sv[t][i] = valid ? sacc[t][i] * a.scale_log2 : -INFINITY;
          mx = fmaxf(mx, sv[t][i]);
        }
      mx = xgroup_max(mx);
      const float mn = fmaxf(m_run, mx);
      const float alpha = exp2f(m_run - mn);
      float ls = 0.f;
#pragma unroll
      for (int t = 0; t < kTiles; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          sv[t][i] = exp2f(sv[t][i] - mn);
          ls += sv[t][i];
        }
      l_run = l_run * alpha + ls;
      m_run = mn;
#pragma unroll
      for (int db = 0; db < 8; ++db) acc[db] *= alpha;

      // O^T += V^T P^T on the matrix cores.  The k-slots 8kg..8kg+7 of a
      // 32-token block are tokens 4kg..4kg+3 of its first tile and of its
      // second tile: exactly the S^T entries this lane holds.
      wave_sync_lds();
#pragma unroll
      for (int kb2 = 0; kb2 < kChunk / 32; ++kb2) {
        float pv[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          pv[i] = sv[2 * kb2][i];
          pv[4 + i] = sv[2 * kb2 + 1][i];
        }
        bf16x8 phi, plo;
        split_bf16x8(pv, phi, plo);
        const uint16_t* r0 = V + (32 * kb2 + 4 * kg + (r16 >> 2)) * kVPitch + 4 * (r16 & 3);
        const uint16_t* r1 = r0 + 16 * kVPitch;
#pragma unroll
        for (int db = 0; db < 8; ++db) {
          const bf16x4 va = lds_read_tr(r0 + 16 * db);
          const bf16x4 vb4 = lds_read_tr(r1 + 16 * db);
          const bf16x8 vA = __builtin_shufflevector(va, vb4, 0, 1, 2, 3, 4, 5, 6, 7);
          acc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vA, phi, acc[db], 0, 0, 0);
          acc[db] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vA, plo, acc[db], 0, 0, 0);
        }
      }
      wave_sync_lds();  // the V tile is rewritten by the next chunk
    }

    // This unit's output: normalised (the whole selection) or a partial.
    // A unit without tokens writes out = 0 and lse = -inf (direct mode); its
    // partials are skipped by the combine.
    const int G = a.G;
    l_run = xgroup_sum(l_run);
    if (r16 < G) {
      if (a.mode == kDirect) {
        const size_t orow = (size_t)cur.lb * a.H_q + (size_t)cur.gv * G + r16;
        const bool any = n_tok > 0;
        const float inv = any ? 1.f / l_run : 0.f;
        float* dst = a.out + orow * kD + 4 * kg;
#pragma unroll
        for (int db = 0; db < 8; ++db)
          *reinterpret_cast<float4*>(dst + 16 * db) =
              make_float4(acc[db][0] * inv, acc[db][1] * inv, acc[db][2] * inv, acc[db][3] * inv);
        if (a.lse && kg == 0) a.lse[orow] = any ? (m_run + log2f(l_run)) * kLn2 : -INFINITY;
      } else if (n_tok > 0) {
        const size_t prow = ((size_t)cur.lb * a.n_split + cur.split) * a.H_q + (size_t)cur.gv * G + r16;
        float* dst = a.part_acc + prow * kD + 4 * kg;
#pragma unroll
        for (int db = 0; db < 8; ++db)
          *reinterpret_cast<float4*>(dst + 16 * db) =
              make_float4(acc[db][0], acc[db][1], acc[db][2], acc[db][3]);
        if (kg == 0) {
          a.part_ml[prow * 2] = m_run;
          a.part_ml[prow * 2 + 1] = l_run;
        }
      }
    }

    if (nitem < 0) break;
    cur = nxt;
    kb = kbn;
    vb = vbn;
    kbf = kbfn;
    vbf = vbfn;
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = qn[s];
    if (!chain && cur.n_tok > 0) {  // not chained (this unit had no tokens): start it cold
      load_v(rows_n, vb, vbf, vraw);
      __builtin_amdgcn_sched_barrier(0);
      load_k(rows_n, kb, kbf, kraw);
      __builtin_amdgcn_sched_barrier(0);
    }
    buf ^= 1;
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
// The splits' (max, sum) pairs and accumulator slices are requested eight at
// a time, all before any is used (one round trip for up to eight splits).
__global__ __launch_bounds__(256) void attn_combine_kernel(CombineArgs a) {
  constexpr int kBatch = 8;
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
  const float2* ml2 = reinterpret_cast<const float2*>(a.part_ml);
  float M = -INFINITY, L = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s0 = 0; s0 < ns; s0 += kBatch) {
    float2 ml[kBatch];
    float4 pa[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {  // clamped: every load is issued
      const size_t row = base + (size_t)min(s0 + u, ns - 1) * a.H_q;
      ml[u] = ml2[row];
      pa[u] = reinterpret_cast<const float4*>(a.part_acc + row * kD)[d4];
    }
    float Mb = M;
#pragma unroll
    for (int u = 0; u < kBatch; ++u)
      if (s0 + u < ns) Mb = fmaxf(Mb, ml[u].x);
    const float r = exp2f(M - Mb);  // earlier batches onto the new maximum (0 at the first)
    L *= r;
    acc.x *= r;
    acc.y *= r;
    acc.z *= r;
    acc.w *= r;
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      if (s0 + u < ns) {
        const float w = exp2f(ml[u].x - Mb);
        L += ml[u].y * w;
        acc.x += pa[u].x * w;
        acc.y += pa[u].y * w;
        acc.z += pa[u].z * w;
        acc.w += pa[u].w * w;
      }
    }
    M = Mb;
  }
  const float inv = 1.f / L;
  *o = make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
  if (a.lse && d4 == 0) a.lse[(size_t)lb * a.H_q + h] = (M + log2f(L)) * kLn2;
}

// Resident wavefront slots the work is sized for: one per SIMD on 256 CUs.
constexpr int64_t kWaveSlots = (int64_t)kWaves * 256;

struct AttnPlan {
  int mode, n_split, split;
};

// Work units are (layer, sequence, KV head, split of the selection).  With at
// least one (layer, sequence, KV head) group per wavefront slot there is no
// split and each unit writes its output (kDirect).  With fewer groups the
// selections are split until there is about one unit per slot, but not below
// kMinSplitTokens (each unit pays a start-up latency and a partial-result
// store; kMinSplitSmall for launches too small to fill the CUs) nor above
// kMaxSplit (the index staging area) (kGlobalPartials).
// Units are numbered KV head fastest, so that the wavefronts of a workgroup
// read the same selected tokens' rows for neighbouring heads at the same time:
// those pieces share DRAM pages.  A split is a whole number of chunks.
// Column groups of at most 16 query heads per KV head.
int attn_col_groups(const Dims& d) { return d.G > 16 ? d.G / 16 : 1; }

// A launch whose units of kMinSplitTokens would not reach one per four CUs
// (a single short layer) is latency-bound: its units may go down to
// kMinSplitSmall tokens, so that more CUs take part.  Launches above that
// keep the larger units, whose start-up cost is then the larger one.
constexpr int kMinSplitSmall = 64;
constexpr int64_t kSmallLaunchUnits = 64;

AttnPlan attn_plan(const Dims& d) {
  const int64_t base = (int64_t)d.n_layers * d.B * d.H_kv * attn_col_groups(d);
  auto round_chunk = [](int64_t t) { return (t + kChunk - 1) / kChunk * kChunk; };
  const int64_t min_split =
      base * ((d.k_max + kMinSplitTokens - 1) / kMinSplitTokens) < kSmallLaunchUnits
          ? kMinSplitSmall
          : kMinSplitTokens;
  int64_t n_split = (kWaveSlots * kSlotUnits + base - 1) / base;
  int64_t split = round_chunk((d.k_max + n_split - 1) / n_split);
  if (split < min_split) split = min_split;
  if (split > kMaxSplit) split = kMaxSplit;
  n_split = (d.k_max + split - 1) / split;
  if (n_split == 1) return {kDirect, 1, (int)round_chunk(d.k_max)};
  return {kGlobalPartials, (int)n_split, (int)split};
}

}  // namespace

int device_cu_count() {
  static const int n = [] {
    int dev = 0, n_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&n_cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        n_cu <= 0)
      n_cu = 256;
    return n_cu;
  }();
  return n;
}

int attn_split_tokens(const Dims& d) { return attn_plan(d).split; }

size_t attn_ws_bytes(const Dims& d) {
  const AttnPlan pl = attn_plan(d);
  if (pl.mode != kGlobalPartials) return 0;
  const size_t rows = (size_t)d.n_layers * d.B * pl.n_split * d.H_q;
  return align_up(sizeof(float) * rows * d.d) + align_up(sizeof(float) * rows * 2);
}

namespace {

template <int KV>
void launch_split(dim3 grid, bool pipe, const AttnArgs& a, hipStream_t s) {
  if (pipe)
    attn_split_kernel<KV, true><<<grid, kWaves * 64, lds_reserve(true), s>>>(a);
  else
    attn_split_kernel<KV, false><<<grid, kWaves * 64, lds_reserve(false), s>>>(a);
}

hipError_t launch_attn_mode(const Dims& d, int kv, const uint16_t* q, const uint16_t* k,
                            const uint16_t* v, const int32_t* idx, uint16_t* kbuf,
                            uint16_t* vbuf, const int32_t* src, const int32_t* fused,
                            const int32_t* counts, float* out, float* lse, void* ws,
                            hipStream_t s) {
  const AttnPlan pl = attn_plan(d);
  // the row staging area holds one split plus a chunk of padding
  if (pl.split > kMaxSplit || pl.split % kChunk != 0) return hipErrorInvalidValue;
  const size_t rows = (size_t)d.n_layers * d.B * pl.n_split * d.H_q;
  float* part_acc = static_cast<float*>(ws);
  float* part_ml = pl.mode == kGlobalPartials
                       ? reinterpret_cast<float*>(static_cast<char*>(ws) +
                                                  align_up(sizeof(float) * rows * d.d))
                       : nullptr;
  const int R = attn_col_groups(d);
  const int64_t n_groups = (int64_t)d.n_layers * d.B * d.H_kv * R;
  const int64_t n_items = n_groups * pl.n_split;
  if (n_items > INT32_MAX / 2) return hipErrorInvalidValue;
  // Work order: the ranges of consecutive units the workgroups own are spread
  // over all (layer, sequence, split) groups by a multiplicative permutation,
  // so that ragged selections even out across workgroups.
  const int n_order = (int)(n_items / (d.H_kv * R));  // (layer, sequence, split) groups
  int perm = 1;
  if (n_order > 2) {
    perm = (int)(0.618 * n_order);
    auto gcd = [](int x, int y) { while (y) { const int t = x % y; x = y; y = t; } return x; };
    while (gcd(perm, n_order) != 1) ++perm;
  }
  AttnArgs a{q, k, v, idx, kbuf, vbuf, src, fused, counts, part_acc, part_ml, out, lse,
             d.kv_stride_layer, d.kv_stride_b, d.B, d.H_q, d.H_kv, d.G / R, d.k_max, d.L_cap,
             pl.n_split, pl.split, (int)n_items, R, pl.mode, n_order, perm, d.n_sets,
             d.scale * kLog2e, 0};
  // One workgroup per CU, fewer only when there are fewer units than CUs:
  // with few units they are spread over all CUs (each CU's share of the
  // bandwidth is limited) rather than packed four to a CU.
  const int n_cu = device_cu_count();
  const dim3 grid((unsigned)(n_items < n_cu ? n_items : n_cu));
  // SPEC_ATTN_SCHEDULE=cold runs every unit from a cold start even where a
  // wavefront takes several (the tests compare both schedules bit for bit).
  const char* sched = getenv("SPEC_ATTN_SCHEDULE");
  const bool force_cold = sched && strcmp(sched, "cold") == 0;
  // some wavefront takes several units: pipeline them
  const bool pipe = !force_cold && n_items > (int64_t)grid.x * kWaves;
  // Sorted order: pipelined, at most one sequence per thread of a workgroup
  // to rank, and at least two groups per workgroup.  SPEC_ATTN_ORDER=perm
  // keeps the permuted order (the tests compare both orders bit for bit).
  const char* order = getenv("SPEC_ATTN_ORDER");
  const bool want_sorted = !(order && strcmp(order, "perm") == 0);
  a.sorted = pipe && want_sorted && d.B <= kSortMaxB && n_order >= 2 * (int64_t)grid.x;
  if (kv == kKvIndexed)
    launch_split<kKvIndexed>(grid, pipe, a, s);
  else if (kv == kKvCompact)
    launch_split<kKvCompact>(grid, pipe, a, s);
  else
    launch_split<kKvElastic>(grid, pipe, a, s);
  if (pl.mode != kGlobalPartials) return hipGetLastError();
  CombineArgs c{part_acc, part_ml, counts, out, lse, d.B, d.H_q, d.k_max, pl.n_split, pl.split};
  const dim3 g2(d.n_layers * d.B, (d.H_q + 7) / 8);
  attn_combine_kernel<<<g2, 256, 0, s>>>(c);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attn(const Dims& d, const uint16_t* q, const uint16_t* k,
                       const uint16_t* v, const int32_t* idx, const int32_t* counts,
                       float* out, float* lse, void* ws, hipStream_t s) {
  return launch_attn_mode(d, idx ? kKvIndexed : kKvCompact, q, k, v, idx, nullptr, nullptr,
                          nullptr, nullptr, counts, out, lse, ws, s);
}

hipError_t launch_attn_elastic(const Dims& d, const uint16_t* q, const uint16_t* k_cache,
                               const uint16_t* v_cache, uint16_t* kbuf, uint16_t* vbuf,
                               const int32_t* slot_src, const int32_t* counts, float* out,
                               float* lse, void* ws, hipStream_t s, const int32_t* fused) {
  return launch_attn_mode(d, kKvElastic, q, k_cache, v_cache, nullptr, kbuf, vbuf, slot_src,
                          fused, counts, out, lse, ws, s);
}

}  // namespace spec
