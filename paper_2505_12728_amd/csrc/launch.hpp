// Host-side launch interfaces between the C ABI layer and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sd {

// ---------------------------------------------------------------- verify
struct VerifyPlan {
  int g;            // query heads per KV head
  int rows;         // k * g query rows that share one KV head
  int row_blocks;   // 16-row blocks per work-group (1..4)
  int row_groups;   // work-groups along the rows of one KV head
  int rows_padded;  // row_groups * row_blocks * 16
  int capacity;     // Lmax or 16 * max_pages
  int keys_per_split;   // fp32 path: keys per split
  int nsplit;           // fp32 path: splits per (sequence, KV head)
  int rows_wg;          // bf16 path: rows per work-group (row_blocks * 16)
  int key_groups;       // bf16 path: wave groups taking alternate tiles
  int stream_wgs;       // bf16 path: grid size (work-groups on the device)
  size_t part_rows;     // rows of partial results in the workspace
  size_t workspace_bytes;
  bool ok;              // false: the shape exceeds the kernels' index range
};

// cus: compute units of the device the call runs on (sizes the bf16 grid)
VerifyPlan plan_verify(int B, int k, int Hq, int Hkv, int D, int capacity, int dtype, int cus);

struct VerifyArgs {
  const void* q;
  const void* kc;
  const void* vc;
  const int32_t* kv_len;
  const int32_t* page_table;
  int max_pages;
  int num_pages;
  int Lmax;
  float* out;
  float* lse;
  int B, k, Hq, Hkv, D;
  float scale;          // score multiplier as given
  float scale_log2;     // scale * log2(e)
  float* part_o;        // [part_rows, D] partial outputs (normalised)
  float* part_lse;      // [part_rows] partial log-sum-exp (log2 units)
  __bf16* out_bf16;     // bf16 stream path: when set, the merge writes out here
                        // as bf16 (and not `out`); used inside the draft layer
};

hipError_t launch_verify(const VerifyArgs& a, const VerifyPlan& p, int dtype, hipStream_t s);

// -------------------------------------------------------------- compress
struct CompressPlan {
  int dh;
  int lat_tile;        // latents per work-group
  int lat_tiles;
  int nsplit;          // splits of the N tokens
  int tokens_per_split;
  size_t workspace_bytes;
};

CompressPlan plan_compress(int B, int N, int C, int d, int H, int dtype, int cus);

struct CompressArgs {
  const void* latents;          // [C, d] bf16 / fp32, or int8 rows (int8 input)
  const void* feats;            // [B, N, d] likewise
  const int8_t* latent_exp;     // int8 input: [C] exponents (row c stands for q * 2^e)
  const int8_t* feat_exp;       // int8 input: [B, N] exponents
  float* out;
  int B, N, C, d, H;
  float scale;
  float scale_log2;
  float* part_o;       // [B, H, nsplit, C, dh]
  float* part_lse;     // [B, H, nsplit, C]
};

// dtype: 0 fp32, 1 bf16, 2 int8 rows with power-of-two row scales
constexpr int kCompressInt8 = 2;
hipError_t launch_compress(const CompressArgs& a, const CompressPlan& p, int dtype, hipStream_t s);
// average pooling of N tokens into C contiguous groups (dtype 0 fp32, 1 bf16)
hipError_t launch_avg_pool(const void* feats, float* out, int B, int N, int C, int d, int dtype, hipStream_t s);

// --------------------------------------------------------------- LM head
struct LmHeadArgs {
  const void* hidden;  // [R, d]
  const void* weight;  // [V, d]
  float* probs;        // [R, V]
  int R, d, V;
  float scale_log2;    // log2(e) / temperature
  float* stats;        // workspace: [R][pairs] (max, sum) pairs, pairs <= ceil(V/16) (per block or per work-group)
  int cus;             // compute units of the device (0: no per-unit balancing)
  int nfull;           // set by the launch: work-groups with a block for every wave (< 0: all)
};

size_t lm_head_workspace_bytes(int R, int V);
hipError_t launch_lm_head(const LmHeadArgs& a, int dtype, hipStream_t s);

// ---------------------------------------------------------------- accept
struct AcceptArgs {
  const float* p;
  const float* q;
  const int32_t* draft;
  const float* u;
  int32_t* n_accepted;
  int32_t* tokens;
  int B, k, V, mode;
};

size_t accept_workspace_bytes(int B, int k, int V, int mode);
hipError_t launch_accept(const AcceptArgs& a, void* workspace, hipStream_t s);
// the same rule with the arrival counters (one uint32 per sequence every
// kCounterStride words, i.e. one per 128-byte line so that the sequences'
// arrivals do not contend for one line; zero on entry, zero again on exit)
// and the chunk partials (accept_partial_bytes) placed apart
constexpr int kCounterStride = 32;
size_t accept_partial_bytes(int B, int k, int V, int mode);
hipError_t launch_accept_split(const AcceptArgs& a, unsigned* counters, void* partials, hipStream_t s);

// acceptance from logits: the rule's fields (p, q, u unused) plus the logits,
// log2(e) / tau and the Philox key / offset of the uniforms
struct AcceptLogitsArgs {
  AcceptArgs rule;
  const void* target_logits;   // [B, k+1, V]
  const void* draft_logits;    // [B, k, V] (sampled mode)
  float scale_log2;
  uint64_t seed, offset;
};

size_t accept_logits_workspace_bytes(int B, int k, int V, int mode);
hipError_t launch_accept_logits(const AcceptLogitsArgs& a, int dtype, void* workspace, hipStream_t s);
hipError_t launch_philox_uniforms(uint64_t seed, uint64_t offset, float* u, int B, int n, hipStream_t s);

// ------------------------------------------------- draft semi-AR layer
constexpr int kLinearRowsPerPass = 128;   // input rows per pass of the weight stream
constexpr int kLinearMaxSplits = 16;      // reduction splits at most

struct LinearArgs {
  const void* x;   // [R, K] bf16
  const void* w;   // [N, K] bf16, or int8 when wscale is set
  float* part;     // [ksplit, R, N] fp32 partial sums
  int R, K, N;
  int ksplit;
  const float* wscale;   // [N] scales of int8 rows, or NULL (bf16 weight)
  int cols;        // output columns per work-group (set from the plan at launch)
};

struct LinearPlan {
  int row_blocks;  // 16-row blocks per pass (1..8)
  int passes;      // passes over the weight (ceil(R / 128))
  int waves;       // waves per work-group
  int cols;        // output columns per work-group: 16 per wave that owns columns
  int ksplit;      // splits of the reduction
  size_t part_bytes;
};

LinearPlan plan_linear(int R, int K, int N, int cus);
hipError_t launch_linear_partial(const LinearArgs& a, const LinearPlan& p, hipStream_t s);
// out = sum of the ksplit partials (+ bias [N]) (+ residual [R, N]), fp32
hipError_t launch_epi_add(const float* part, int ksplit, int R, int N, const float* bias,
                          const float* residual, float* out, hipStream_t s);

struct SemiArArgs {
  const void* u;       // [B r, 2d] bf16: concat(F_T, E) of the new rows
  const void* fc_w;    // [d, 2d] bf16
  const float* fc_b;   // [d]
  const float* ln1;    // [d]
  const void* wqkv;    // [(Hq + 2 Hkv) D, d] bf16
  const void* wo;      // [d, Hq D] bf16
  const float* ln2;    // [d]
  const void* wgu;     // [2I, d] bf16
  const void* wdown;   // [d, I] bf16
  // int8 draft: the five weights above hold int8 rows and these their
  // per-row scales (all NULL for the bf16 draft)
  const float* fc_s;
  const float* wqkv_s;
  const float* wo_s;
  const float* wgu_s;
  const float* wdown_s;
  void* k_cache;       // [B, Lmax, Hkv, D] bf16
  void* v_cache;
  const int32_t* pos;  // [B] first new position of each sequence
  float* out;          // [B r, d]
  int B, r, d, Hq, Hkv, I, Lmax;
  float eps, theta;
  void* workspace;
};

struct SemiArPlan {
  LinearPlan fc, qkv, o, gu, down;
  VerifyPlan verify;
  size_t off_part, off_x0, off_h, off_q, off_attn16, off_x1, off_act, off_kvlen, off_ss, off_verify;
  size_t workspace_bytes;
  bool ok;
};

SemiArPlan plan_semi_ar(int B, int r, int d, int Hq, int Hkv, int I, int Lmax, int cus);
hipError_t launch_semi_ar(const SemiArArgs& a, const SemiArPlan& p, hipStream_t s);

// K drafts in K / kp passes: pass 0 on layer.u (layer.r rows, the last kp
// placeholders), later passes on 2 kp rows built on the device
struct SemiArDraftArgs {
  SemiArArgs layer;      // layer.out and layer.workspace are set per pass
  const void* lm_w;      // [V, d] bf16
  const void* emb;       // [V, d] bf16
  const void* ph;        // [2d] bf16 placeholder input
  const float* u;        // [B, K]
  int32_t* tokens;       // [B, K]
  float* q;              // [B, K, V]
  int V, K, kp;
  float temperature;
  void* workspace;
};

struct SemiArDraftPlan {
  SemiArPlan first, later;
  size_t off_layer, off_out, off_unext, off_hid, off_probs, off_lmstats, off_sample, off_nacc, off_ut, off_tok,
      off_pos;
  size_t workspace_bytes;
  int cus;
  bool ok;
};

SemiArDraftPlan plan_semi_ar_draft(int B, int r0, int d, int Hq, int Hkv, int I, int Lmax, int V, int K, int kp,
                                   int cus);
hipError_t launch_semi_ar_draft(const SemiArDraftArgs& a, const SemiArDraftPlan& p, hipStream_t s);

}  // namespace sd
