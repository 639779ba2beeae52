// Device-side argument blocks and launch entry points of the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "simsd_plan.h"

namespace simsd {

struct AttnArgs {
  const void* q;
  const void* k_new;
  const void* v_new;
  const void* k_cache;
  const void* v_cache;
  const int32_t* block_table;
  const int32_t* prefix_lens;
  const int32_t* step_map;
  const int32_t* num_ref;
  void* out;
  float* lse;
  float* part;        // split partials (workspace), or null when splits == 1
  int64_t* stream_seq0; // stream decomposition: per-sequence tile offsets (workspace)
  int64_t cs_seq, cs_tok, cs_head;
  int batch, hq, hkv, group, B, L, n_new, rows, rows_pb, row_blocks;
  int page_size, max_pages, chunk, splits, max_prefix;
  int stream_groups;  // stream decomposition: work-groups (0 = chunked decomposition)
  float scale_log2;
  int rope;           // rotary embedding of the new slots' q and k at the RoPE-copy positions
  float rope_step;    // pair i turns by pos * exp2(i * rope_step)
  float rope_theta;   // the base itself (the fp32 path forms its angles in fp64)
};

struct AcceptArgs {
  // Greedy and sampled (the greedy kernels read only this first block, so it
  // stays small and in one place for their argument loads).
  const void* logits;
  const int32_t* draft_ids;
  const int32_t* step_map;
  const int32_t* num_ref;
  int32_t* target_ids;
  float* confidence;
  float* draft_prob;          // greedy: target probability of each draft; sampled: p_theta(D_r)
  int32_t* accept_len;
  AcceptPartial* part;
  int64_t nvec, chunk_vecs;
  int B, L, V, cpr;
  int rows;                   // partial rows per sequence: B, or B + L (sampled)
  float cl;                   // log2(e) / temperature
  // Sampled only.
  const void* draft_logits;   // [batch, L, V], same dtype as logits
  const float* uniforms;      // [batch, L + 1]
  float* p_draft;             // p_phi(D_r)
  int32_t* correction;        // token drawn at the first rejection, or -1
  DrawRow* draw_row;          // [batch]
  DrawPartial* draw_part;     // [batch, draw_chunks]
  int64_t draw_vecs;
  int draw_chunks;
  const float* xdraft;        // LM-head path: the drafted tokens' logits [batch, L]
};

// LM-head product fused with the vocabulary scan.
struct LmheadArgs {
  const void* hidden;         // [R = batch * B, H] bf16
  const void* weight;         // [V, H] bf16
  const int32_t* draft_ids;
  const int32_t* step_map;
  const int32_t* num_ref;
  AcceptPartial* part;        // [R, vtiles]
  AcceptPartial* merged;      // [R]: the partials of each row merged
  float* xdraft;              // [batch, L]
  int R, B, L, V, H, vtiles;
};

hipError_t launch_attention(const simsd_attn_desc& d, const AttnPlan& p, const AttnArgs& a,
                            hipStream_t stream);
hipError_t launch_accept(const simsd_accept_desc& d, const AcceptPlan& p, const AcceptArgs& a,
                         hipStream_t stream);
hipError_t launch_accept_sampled(const simsd_accept_desc& d, const AcceptPlan& p,
                                 const AcceptArgs& a, hipStream_t stream);
hipError_t launch_lmhead_scan(const LmheadArgs& a, hipStream_t stream);
hipError_t launch_lmhead_merge(const LmheadArgs& a, hipStream_t st);
hipError_t launch_finalize_lmhead(int batch, const AcceptArgs& a, hipStream_t stream);
int lmhead_vocab_tile(int rows);   // vocabulary entries per scan work-group, by row count
// Device of `stream` (a hipStream_t; NULL = the current device) and its
// compute units, queried once per device; on failure *cus is an MI355X's 256
// and the error is returned for the caller to report after validation.
hipError_t stream_device(void* stream, int* dev, int* cus);
int lmhead_stage();        // reduction elements per stage (H must be a multiple)

}  // namespace simsd
