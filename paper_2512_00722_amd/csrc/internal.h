// Internal host-side interface between the C ABI layer and the kernel files.
// Nothing here is exported from the shared library.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace spec {

// Dimensions after validation, with defaults resolved and derived values.
struct Dims {
  int B, L_cap, L_max, k_max;
  int H_r, d_r;
  int n_layers, H_q, H_kv, d, G;
  int n_sets;  // token sets per sequence: 1 (summed heads) or H_kv (one per KV head)
  int64_t kr_stride_b, kv_stride_layer, kv_stride_b;
  float scale_r, scale;
};

// ---- workspace geometry (every region aligned to 256 bytes) -------------
constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Retrieval scoring: tokens per workgroup of the logits kernel, 256, halved
// (down to 64) while the grid would have fewer workgroups than the chip has
// CUs: a short single sequence is latency-bound, and more, smaller blocks
// keep more bytes in flight.
constexpr int kScoreTokensPerBlock = 256;
constexpr int kScoreTokensPerBlockMin = 64;
constexpr int64_t kScoreMinBlocks = 256;
// Softmax/head-sum kernel: tokens per workgroup.
constexpr int kSoftTokensPerBlock = 1024;

inline int score_tokens_per_block(const Dims& d) {
  int tpb = kScoreTokensPerBlock;
  while (tpb > kScoreTokensPerBlockMin &&
         (int64_t)d.B * ((d.L_max + tpb - 1) / tpb) < kScoreMinBlocks)
    tpb /= 2;
  return tpb;
}
inline int score_blocks(const Dims& d) {
  const int tpb = score_tokens_per_block(d);
  return (d.L_max + tpb - 1) / tpb;
}
// Top-k: 4096-bin histogram of the top 12 bits of the score keys per score
// row (B * n_sets rows).
constexpr int kTopkBins = 4096;
inline size_t topk_hist_bytes(const Dims& d) {
  return align_up(sizeof(int32_t) * (size_t)d.B * d.n_sets * kTopkBins);
}

// logits [B][L_max][H_r] fp32 + per-block (max, sum) [B][n_blk][H_r][2] fp32
// + the top-k histogram of the scores written.
inline size_t score_logits_bytes(const Dims& d) {
  return align_up(sizeof(float) * (size_t)d.B * d.L_max * d.H_r);
}
inline size_t score_part_bytes(const Dims& d) {
  return align_up(sizeof(float) * 2 * (size_t)d.B * score_blocks(d) * d.H_r);
}
inline size_t score_ws_bytes(const Dims& d) {
  return score_logits_bytes(d) + score_part_bytes(d) + topk_hist_bytes(d);
}
// The regions of a score workspace: logits, per-block pairs, histogram.
inline float* score_ws_logits(void* ws) { return static_cast<float*>(ws); }
inline float* score_ws_part(const Dims& d, void* ws) {
  return reinterpret_cast<float*>(static_cast<char*>(ws) + score_logits_bytes(d));
}
inline int32_t* score_ws_hist(const Dims& d, void* ws) {
  return reinterpret_cast<int32_t*>(static_cast<char*>(ws) + score_logits_bytes(d) +
                                    score_part_bytes(d));
}

// Short score rows are normalised, summed and selected by one workgroup each,
// their keys held in LDS (one launch in place of the softmax and the two
// tiled selection kernels): rows of at most kRowSelectMaxL tokens whose
// logits (heads per row x tokens) number at most kRowSelectMaxLogits.  One
// workgroup streams only a few tens of GB/s, so longer rows are faster on
// the tiled path, which spreads a row over many workgroups.
constexpr int kRowSelectMaxL = 8192;
constexpr int64_t kRowSelectMaxLogits = 32768;
// heads_per_row: H_r / n_sets for the fused step, 1 for a standalone
// selection.  SPEC_TOPK_PATH=tiles in the environment forces the tiled
// kernels (tests compare both paths).
bool row_select_fits(const Dims& d, int heads_per_row);

// Per-tile lists of the selection (tokens per tile: kTopkTile): the
// threshold bin of each row, per-tile counts, the tokens above the threshold
// bin, and the bin's candidates (key, token).
constexpr int kTopkTile = 2048;
inline int topk_tiles(const Dims& d) { return (d.L_max + kTopkTile - 1) / kTopkTile; }
inline size_t topk_lists_bytes(const Dims& d) {
  const size_t rows = (size_t)d.B * d.n_sets;
  const size_t n = rows * topk_tiles(d);
  return align_up(sizeof(int32_t) * 4 * rows) + align_up(sizeof(int32_t) * 2 * n) +
         3 * align_up(sizeof(int32_t) * n * kTopkTile);
}
inline size_t topk_ws_bytes(const Dims& d) { return topk_hist_bytes(d) + topk_lists_bytes(d); }

// Attention: tokens of the selection per work unit, and the workspace for
// partial results (zero unless a selection is split across workgroups).
int attn_split_tokens(const Dims& d);
size_t attn_ws_bytes(const Dims& d);

// Elastic loading: per sequence the list of (slot, token) copies, then per
// sequence whether the attention loads its rows itself (the fused step).
inline size_t delta_ws_bytes(const Dims& d) {
  return align_up(sizeof(int32_t) * 2 * (size_t)d.B * d.k_max) +
         align_up(sizeof(int32_t) * (size_t)d.B);
}
inline int32_t* delta_ws_fused(const Dims& d, void* ws) {
  return reinterpret_cast<int32_t*>(static_cast<char*>(ws) +
                                    align_up(sizeof(int32_t) * 2 * (size_t)d.B * d.k_max));
}
// The fused step's elastic attention loads a sequence's new rows itself
// when more than this share (percent) of its selection is new, as in a full
// reload; otherwise the rows are copied first and the attention only reads.
// A kernel that writes while it streams runs at ~4.8 TB/s, one that only
// reads at ~6.3, so the copy wins for small updates.
constexpr int kElasticFusePct = 50;

// Retrieval-head front end: embedding width, vocabulary and the rotary /
// YaRN parameters, validated (alpha < beta; orig_ctx > 0 when scale > 1).
struct FrontDims {
  int vocab, hidden;
  float base, scale, alpha, beta;
  int orig_ctx;
};
// The projection splits the hidden dimension over at most this many
// workgroups per output tile; the workspace holds the rotary frequency table
// and one fp32 partial result [split][B][2 * H_r * d_r] per split.
constexpr int kFrontMaxSplit = 16;
size_t front_ws_bytes(const Dims& d);

// MLA sparse decode attention: d_c = 512, d_rope = 64, d_nope = d_v = 128
// (validated), H in {64, 128}; the latent cache rows are d_c + d_rope wide.
struct MlaDims {
  int B, L_cap, k_max, n_layers, H;
  int64_t stride_layer, stride_b;  // elements between layers / sequences of the cache
  float scale;                     // resolved: 1/sqrt(d_nope + d_rope) by default
};
size_t mla_ws_bytes(const MlaDims& d);

// The allocation-free decode step keeps its workspace in a static device
// array of this size (one per GPU, held until the process ends);
// static_scratch() gives its device address on the current GPU.
constexpr size_t kStaticScratchBytes = size_t(64) << 20;
hipError_t static_scratch(void** out);

// Compute units of the device the process first launches on, queried once
// and cached (kernels size their grids with it; every grid size is correct,
// so the launch path makes no device query).
int device_cu_count();

// ---- launchers (return the HIP launch status) --------------------------
hipError_t launch_score(const Dims& d, const uint16_t* q_r, const uint16_t* k_r,
                        const int32_t* seq_lens, float* scores, void* ws,
                        hipStream_t s);
// The logits kernel alone (logits and per-block pairs into the score
// workspace); zero_hist: also clear the selection histogram there.
hipError_t launch_logits(const Dims& d, const uint16_t* q_r, const uint16_t* k_r,
                         const int32_t* seq_lens, void* ws, bool zero_hist, hipStream_t s);
// One workgroup per score row (requires row_select_fits): from the logits
// and pairs of the score workspace `ws_score` (scores written to `scores`
// when not null), or, with ws_score null, from the scores in `scores`.
hipError_t launch_row_select(const Dims& d, void* ws_score, float* scores,
                             const int32_t* seq_lens, const int32_t* ks, int32_t* idx,
                             int32_t* counts, hipStream_t s);
// Scores and selection of the fused step: the row kernel where it fits,
// else the score kernels and the tiled selection.  scores_keep: where the
// caller wants the scores (may be null); scores_ws: a [B][n_sets][L_max]
// fp32 buffer for the tiled path.
hipError_t launch_score_select(const Dims& d, const uint16_t* q_r, const uint16_t* k_r,
                               const int32_t* seq_lens, const int32_t* ks, float* scores_keep,
                               float* scores_ws, int32_t* idx, int32_t* counts, void* ws_score,
                               void* ws_topk, hipStream_t s);
hipError_t launch_topk(const Dims& d, const float* scores, const int32_t* seq_lens,
                       const int32_t* ks, int32_t* idx, int32_t* counts, void* ws,
                       hipStream_t s);
// Selection only, from a histogram already built over the same scores.
hipError_t launch_topk_select(const Dims& d, const float* scores, const int32_t* seq_lens,
                              const int32_t* ks, const int32_t* hist, void* lists, int32_t* idx,
                              int32_t* counts, hipStream_t s);
hipError_t launch_gather(const Dims& d, const uint16_t* k_cache, const uint16_t* v_cache,
                         const int32_t* idx, const int32_t* counts, uint16_t* k_sel,
                         uint16_t* v_sel, hipStream_t s);
hipError_t launch_attn(const Dims& d, const uint16_t* q, const uint16_t* k,
                       const uint16_t* v, const int32_t* idx, const int32_t* counts,
                       float* out, float* lse, void* ws, hipStream_t s);
// Attention over the slot buffers after an elastic update: slots with
// slot_src[b][slot] >= 0 are read from the caches at that token and written
// into the slot on the way; the others are read from the slot.
// fused (nullable, [B]): only sequences with fused[b] != 0 load rows from
// the caches; the others are read from their slots throughout.
hipError_t launch_attn_elastic(const Dims& d, const uint16_t* q, const uint16_t* k_cache,
                               const uint16_t* v_cache, uint16_t* kbuf, uint16_t* vbuf,
                               const int32_t* slot_src, const int32_t* counts, float* out,
                               float* lse, void* ws, hipStream_t s,
                               const int32_t* fused = nullptr);
hipError_t launch_delta(const Dims& d, const int32_t* idx_now, const int32_t* counts,
                        const uint16_t* k_cache, const uint16_t* v_cache,
                        int32_t* slot_tok, int32_t* slot_src, uint16_t* kbuf, uint16_t* vbuf,
                        int32_t* n_changed, void* ws, hipStream_t s);
// Elastic loading in two parts: the slot plan (the (slot, token) list in
// ws; slot_src: per slot the token loaded into it, or -1), then the copy of
// the listed rows of n_layers layers from a source cache (device memory, or
// pinned host memory through its device address) into the slot buffers.
// fuse_pct >= 0: also mark, in ws, the sequences more than fuse_pct % of
// whose selection is new (the attention loads their rows; the copy skips
// them).
hipError_t launch_delta_plan(const Dims& d, const int32_t* idx_now, const int32_t* counts,
                             int32_t* slot_tok, int32_t* slot_src, int32_t* n_changed, void* ws,
                             hipStream_t s, int fuse_pct = -1);
// from_host: the source rows are in pinned host memory (the host-offloaded
// layers); device-to-device copies run fewer workgroups per CU.
hipError_t launch_delta_copy(const Dims& d, const uint16_t* k_src, const uint16_t* v_src,
                             int64_t src_stride_layer, int64_t src_stride_b, int n_layers,
                             const int32_t* n_changed, uint16_t* kbuf, uint16_t* vbuf,
                             const void* ws, hipStream_t s, const int32_t* skip = nullptr,
                             bool from_host = false);
hipError_t launch_mla(const MlaDims& d, const uint16_t* q, const uint16_t* ckv,
                      const uint16_t* w_uk, const uint16_t* w_uv, const int32_t* idx,
                      const int32_t* counts, float* out, float* lse, void* ws, hipStream_t s);
hipError_t launch_retrieval_qk(const Dims& d, const FrontDims& f, const int32_t* tokens,
                               const int32_t* pos, const uint16_t* emb, const uint16_t* w_q,
                               const uint16_t* w_k, uint16_t* q_r, uint16_t* k_r, void* ws,
                               hipStream_t s);

}  // namespace spec
