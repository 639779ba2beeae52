// Launch planning and argument checking for the SimSD verification step.
// Pure host C++ (no HIP): every decision here is testable without a GPU.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>

#include "simsd.h"

namespace simsd {

constexpr int kTile = 64;            // keys per attention tile
constexpr int kMaxNew = 64;          // B + L limit (one 64-bit visibility word per row)
constexpr int kMaxGroup = 16;        // Hq / Hkv limit
constexpr int kStreamChunk = -1;    // kv_chunk value that asks for the stream decomposition
constexpr int kMaxStreamBatch = 256;  // stream decomposition: largest batch
constexpr int kMinAutoChunk = 64;   // shortest automatic prefix chunk (keys)
constexpr int kMaxAutoChunk = 8192;  // longest automatic prefix chunk (keys)
constexpr int kAcceptThreads = 256;  // threads of the vocabulary-scan work-group
constexpr int kAcceptPerCU = 2;     // scan work-groups per compute unit the chunk heuristic aims for

struct AttnPlan {
  int group = 0;        // Hq / Hkv
  int n_new = 0;        // B + L
  int rows = 0;         // M = group * n_new packed query rows per (sequence, KV head)
  int waves = 0;        // waves per work-group
  int row_waves = 0;    // waves that own distinct rows (bf16: 32 rows each)
  int rows_pb = 0;      // rows per work-group (row block)
  int row_blocks = 0;   // ceil(rows / rows_pb)
  int chunk = 0;        // prefix keys per split
  int splits = 0;       // grid.x: ceil(max_prefix_len / chunk), >= 1
  bool stream = false;  // bf16: stream decomposition (equal tile ranges per work-group)
  int stream_groups = 0;
  int64_t pairs = 0;    // batch * Hkv * row_blocks
  size_t part_floats = 0;   // floats per split partial: rows_pb * (head_dim + 2)
  size_t workspace = 0;     // total bytes
  float scale_log2 = 0.f;   // softmax scale * log2(e)
  float rope_step = 0.f;    // rotary: log2 of the frequency ratio between pairs (0 = off)
};

struct AcceptPlan {
  int rows = 0;           // partial rows per sequence: B (greedy) or B + L (sampled)
  int draw_chunks = 0;    // sampled: vocabulary chunks of the residual draw per sequence
  int64_t draw_vecs = 0;  // sampled: vectors per draw chunk
  size_t draw_row_off = 0;   // sampled: workspace offsets (bytes) of the per-sequence
  size_t draw_part_off = 0;  //   draw rows and of the draw chunk partials
  int vec = 1;            // elements per vector load (16 bytes), or 1 for the scalar path
  int64_t nvec = 0;       // vectors per row
  int cpr = 0;            // chunks (work-groups) per row
  int64_t chunk_vecs = 0; // vectors per chunk
  size_t workspace = 0;
};

// Partial result of one vocabulary chunk: max, lowest index reaching it,
// sum of exp(x - max).
struct AcceptPartial {
  float mx;
  int32_t ix;
  float sm;
  int32_t pad;
};

struct LmheadPlan {
  int vtiles = 0;         // vocabulary tiles (scan work-groups per row tile)
  size_t merged_off = 0;  // workspace offset (bytes) of the merged per-row partials
  size_t xdraft_off = 0;  // workspace offset (bytes) of the drafted tokens' logits
  size_t workspace = 0;
};

// Sampled rule: what the draw needs of one sequence (written once the
// acceptance is decided; acc >= gamma, kr = -1 when every draft was accepted).
struct DrawRow {
  int32_t acc, kr;
  float mt, ct, md, cd;   // row maxima and reciprocal sums of the two rows
  int32_t pad[2];
};

// Sampled rule: one vocabulary chunk of the draw row: sums of the residual
// and of p_theta, and the last index of each with positive weight.
struct DrawPartial {
  float sq, st;
  int32_t lq, lt;
};

void set_error(const std::string& msg);

// `cus`: compute units of the device the call runs on (it sizes the grids and
// the stream decomposition's workspace); must be >= 1.
simsd_status plan_attention(const simsd_attn_desc* d, int cus, AttnPlan* p);
simsd_status check_attention_args(const simsd_attn_desc* d, const AttnPlan& p, const void* q,
                                  const void* k_new, const void* v_new, const void* k_cache,
                                  const void* v_cache, const int32_t* block_table,
                                  const int32_t* prefix_lens, const int32_t* step_map,
                                  const int32_t* num_ref, const void* out, const float* lse,
                                  const void* workspace, size_t workspace_bytes);

// sampled: the stochastic entry point, whose scan also covers the L draft rows.
simsd_status plan_accept(const simsd_accept_desc* d, int cus, AcceptPlan* p, bool sampled = false);
// The accept arguments other than the workspace.
simsd_status check_accept_inputs(const simsd_accept_desc* d, const void* logits,
                                 const int32_t* draft_ids, const int32_t* step_map,
                                 const int32_t* num_ref, const int32_t* target_ids,
                                 const int32_t* accept_len);
simsd_status check_accept_args(const simsd_accept_desc* d, const AcceptPlan& p,
                               const void* logits, const int32_t* draft_ids,
                               const int32_t* step_map, const int32_t* num_ref,
                               const int32_t* target_ids, const float* confidence,
                               const float* draft_prob, const int32_t* accept_len,
                               const void* workspace, size_t workspace_bytes);
simsd_status plan_lmhead(const simsd_lmhead_desc* d, int vocab_tile, int stage, LmheadPlan* p);
simsd_status check_lmhead_args(const simsd_lmhead_desc* d, const LmheadPlan& p, const void* hidden,
                               const void* weight, const int32_t* draft_ids,
                               const int32_t* step_map, const int32_t* num_ref,
                               const int32_t* target_ids, const int32_t* accept_len,
                               const void* workspace, size_t workspace_bytes);
simsd_status check_accept_sampled_args(const simsd_accept_desc* d, const AcceptPlan& p,
                                       float temperature, const void* logits,
                                       const void* draft_logits, const int32_t* draft_ids,
                                       const int32_t* step_map, const int32_t* num_ref,
                                       const float* uniforms, const int32_t* accept_len,
                                       const int32_t* correction, const void* workspace,
                                       size_t workspace_bytes);

}  // namespace simsd
