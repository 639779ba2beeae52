// Launch planning, argument checking and the host-only helpers of the C ABI.
// No HIP calls: this file is plain C++17.
#include "simsd_plan.h"

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <string>

namespace simsd {

static thread_local std::string g_last_error;

void set_error(const std::string& msg) { g_last_error = msg; }

static simsd_status fail(simsd_status st, const std::string& msg) {
  set_error(msg);
  return st;
}

static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

static int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

static int elem_bytes(simsd_dtype t) { return t == SIMSD_F32 ? 4 : 2; }

// A dtype field as the integer a C caller stored there.  Reading the enum
// itself would be undefined for a value outside the enumeration, which the
// ABI must reject rather than trust.
static_assert(sizeof(simsd_dtype) == sizeof(int), "simsd_dtype is int-sized");
static int dtype_code(const simsd_dtype& field) {
  int v;
  std::memcpy(&v, &field, sizeof v);
  return v;
}
static bool known_dtype(const simsd_dtype& field) {
  const int v = dtype_code(field);
  return v == SIMSD_F32 || v == SIMSD_BF16;
}

simsd_status plan_attention(const simsd_attn_desc* d, int cus, AttnPlan* p) {
  if (!d || !p) return fail(SIMSD_ERR_NULL_POINTER, "attention: descriptor is NULL");
  if (cus < 1) return fail(SIMSD_ERR_HIP, "attention: the device reports no compute units");
  if (!known_dtype(d->dtype))
    return fail(SIMSD_ERR_UNSUPPORTED, "attention: dtype must be SIMSD_F32 or SIMSD_BF16");
  if (d->batch < 1 || d->batch > 65535)
    return fail(SIMSD_ERR_BAD_SHAPE, "attention: batch must be in [1, 65535]");
  if (d->num_q_heads < 1 || d->num_kv_heads < 1 || d->num_q_heads % d->num_kv_heads != 0)
    return fail(SIMSD_ERR_BAD_SHAPE,
                "attention: need num_q_heads, num_kv_heads >= 1 and Hq % Hkv == 0");
  if (d->num_q_heads / d->num_kv_heads > kMaxGroup)
    return fail(SIMSD_ERR_UNSUPPORTED, "attention: Hq / Hkv must be <= 16");
  if (d->head_dim != 64 && d->head_dim != 128)
    return fail(SIMSD_ERR_UNSUPPORTED, "attention: head_dim must be 64 or 128");
  if (d->block_size < 1 || d->max_ref < 0 || d->max_ref > d->block_size ||
      int64_t{d->block_size} + d->max_ref > kMaxNew)
    return fail(SIMSD_ERR_BAD_SHAPE,
                "attention: need block_size >= 1, 0 <= max_ref <= block_size, "
                "block_size + max_ref <= 64");
  if (d->max_prefix_len < 0) return fail(SIMSD_ERR_BAD_SHAPE, "attention: max_prefix_len < 0");
  if (d->page_size < 0) return fail(SIMSD_ERR_BAD_SHAPE, "attention: page_size < 0");
  if (d->page_size > 0 && d->max_pages_per_seq < ceil_div(d->max_prefix_len, d->page_size))
    return fail(SIMSD_ERR_BAD_SHAPE,
                "attention: max_pages_per_seq < ceil(max_prefix_len / page_size)");
  if (d->kv_chunk < kStreamChunk || (d->kv_chunk > 0 && d->kv_chunk % kTile != 0))
    return fail(SIMSD_ERR_BAD_SHAPE,
                "attention: kv_chunk must be -1 (stream), 0 (auto) or a multiple of 64");
  const int eb = elem_bytes(d->dtype);
  const int64_t strides[3] = {d->cache_stride_seq, d->cache_stride_token, d->cache_stride_head};
  for (int64_t s : strides) {
    if (s < 0) return fail(SIMSD_ERR_BAD_SHAPE, "attention: negative cache stride");
    // s * eb a multiple of 16 bytes, tested without forming the product
    if (s % (16 / eb) != 0)
      return fail(SIMSD_ERR_ALIGNMENT, "attention: cache strides must be multiples of 16 bytes");
    if (s > (int64_t{1} << 48))
      return fail(SIMSD_ERR_BAD_SHAPE, "attention: cache stride beyond 2^48 elements");
  }
  if (!(std::isfinite(d->scale) && d->scale >= 0.f))
    return fail(SIMSD_ERR_BAD_SHAPE, "attention: scale must be finite and >= 0");
  if (!(std::isfinite(d->rope_theta) && d->rope_theta >= 0.f))
    return fail(SIMSD_ERR_BAD_SHAPE, "attention: rope_theta must be finite and >= 0");

  AttnPlan r;
  r.group = d->num_q_heads / d->num_kv_heads;
  r.n_new = d->block_size + d->max_ref;
  r.rows = r.group * r.n_new;
  if (d->dtype == SIMSD_BF16) {
    // One 32-row MFMA block per row wave; a power of two in [2, 8].  Two row
    // waves are each paired with a second wave taking the other half of
    // every key tile (4 waves per group, two groups per CU); four or eight
    // row waves take whole tiles (one group per CU).  (Four row waves with
    // half tiles, 8 waves, measured 7-9 % slower on the SDAR-8B layer: one
    // 32-key block per wave between barriers.  The rotary variant keeps them:
    // the whole-tile one needs more registers than its bound allows.)
    const int need = static_cast<int>(ceil_div(std::min(r.rows, 256), 32));
    r.row_waves = 2;
    while (r.row_waves < need) r.row_waves *= 2;
    r.waves = r.row_waves <= 2 ? 2 * r.row_waves : r.row_waves;
    r.rows_pb = r.row_waves * 32;
  } else {
    r.waves = 4;          // 8 rows per wave, one wave per row at a time
    r.row_waves = 4;
    r.rows_pb = 32;
  }
  r.row_blocks = static_cast<int>(ceil_div(r.rows, r.rows_pb));
  if (static_cast<int64_t>(d->num_kv_heads) * r.row_blocks > 65535)
    return fail(SIMSD_ERR_BAD_SHAPE, "attention: num_kv_heads * row blocks exceeds 65535");
  r.pairs = static_cast<int64_t>(d->batch) * d->num_kv_heads * r.row_blocks;
  if (d->kv_chunk > 0) {
    r.chunk = d->kv_chunk;
  } else {
    // Split the longest prefix so that about as many work-groups exist as the
    // chip holds at once: one group per CU, two for the two-row-wave groups.
    const int64_t target = r.row_waves >= 4 ? cus : 2 * int64_t{cus};
    int64_t c = ceil_div(static_cast<int64_t>(d->max_prefix_len) * r.pairs, target);
    c = ceil_div(c, kTile) * kTile;
    if (c < kMinAutoChunk) c = kMinAutoChunk;
    if (c > kMaxAutoChunk) c = kMaxAutoChunk;
    r.chunk = static_cast<int>(c);
  }
  r.splits = d->max_prefix_len > 0 ? static_cast<int>(ceil_div(d->max_prefix_len, r.chunk)) : 1;
  if (r.splits > 65535 * 1024) return fail(SIMSD_ERR_BAD_SHAPE, "attention: too many splits");
  r.part_floats = static_cast<size_t>(r.rows_pb) * (d->head_dim + 2);
  r.workspace = r.splits > 1 ? static_cast<size_t>(r.pairs) * r.splits * r.part_floats * 4 : 0;
  // Large bf16 problems take the stream decomposition: one work-group per
  // resident slot, each with an equal share of all tiles (ragged prefixes do
  // not unbalance it).  It is chosen when the chunked grid would take more than
  // one round of resident groups (where ragged prefixes leave slots idle) and
  // there are at least 8 tiles per group; kv_chunk -1 asks for it at any size.  Workspace: two partial slots per group, then the
  // per-sequence tile offsets.  (Row blocks of up to 128 rows; the 8-wave
  // 256-row group keeps the chunks.)
  const bool can_stream = d->dtype == SIMSD_BF16 && d->batch <= kMaxStreamBatch &&
                          r.row_waves <= 4;
  if (d->kv_chunk == kStreamChunk && !can_stream)
    return fail(SIMSD_ERR_UNSUPPORTED,
                "attention: kv_chunk -1 (stream) needs bf16, at most 128 packed rows "
                "(Hq/Hkv * (B + L)) and batch <= 256");
  if (can_stream && d->kv_chunk <= 0) {
    // Stream groups: 8 waves (one per CU) for four row waves, else 4 (two per CU).
    const int64_t groups = r.row_waves >= 4 ? cus : 2 * int64_t{cus};
    const int64_t tiles = r.pairs * (ceil_div(d->max_prefix_len, kTile) + 1);
    if (d->kv_chunk == kStreamChunk || (tiles >= 8 * groups && r.pairs * r.splits > groups)) {
      r.stream = true;
      r.stream_groups = static_cast<int>(groups);
      r.workspace = static_cast<size_t>(groups) * 2 * r.part_floats * 4 +
                    static_cast<size_t>(kMaxStreamBatch + 1) * 8;
    }
  }
  const float scale = d->scale > 0.f ? d->scale : 1.0f / std::sqrt(static_cast<float>(d->head_dim));
  r.scale_log2 = scale * 1.4426950408889634f;
  // theta^(-2i/d) = exp2(i * rope_step), rope_step = -2 log2(theta) / d
  r.rope_step = d->rope_theta > 0.f ? -2.0f * std::log2(d->rope_theta) / d->head_dim : 0.f;
  *p = r;
  return SIMSD_OK;
}

simsd_status check_attention_args(const simsd_attn_desc* d, const AttnPlan& p, const void* q,
                                  const void* k_new, const void* v_new, const void* k_cache,
                                  const void* v_cache, const int32_t* block_table,
                                  const int32_t* prefix_lens, const int32_t* step_map,
                                  const int32_t* num_ref, const void* out, const float* lse,
                                  const void* workspace, size_t workspace_bytes) {
  if (!q || !k_new || !v_new || !prefix_lens || !step_map || !num_ref || !out)
    return fail(SIMSD_ERR_NULL_POINTER,
                "attention: q, k_new, v_new, prefix_lens, step_map, num_ref and out are required");
  if (d->max_prefix_len > 0 && (!k_cache || !v_cache))
    return fail(SIMSD_ERR_NULL_POINTER, "attention: k_cache/v_cache required when max_prefix_len > 0");
  if (d->page_size > 0 && d->max_prefix_len > 0 && !block_table)
    return fail(SIMSD_ERR_NULL_POINTER, "attention: block_table required for a paged cache");
  const void* aligned[] = {q, k_new, v_new, out};
  for (const void* a : aligned)
    if (!aligned16(a)) return fail(SIMSD_ERR_ALIGNMENT, "attention: q/k_new/v_new/out must be 16-byte aligned");
  if (d->max_prefix_len > 0 && (!aligned16(k_cache) || !aligned16(v_cache)))
    return fail(SIMSD_ERR_ALIGNMENT, "attention: k_cache/v_cache must be 16-byte aligned");
  if (lse && (reinterpret_cast<uintptr_t>(lse) & 3u))
    return fail(SIMSD_ERR_ALIGNMENT, "attention: lse must be 4-byte aligned");
  if (p.workspace > 0) {
    if (!workspace) return fail(SIMSD_ERR_WORKSPACE, "attention: workspace is NULL");
    if (!aligned16(workspace)) return fail(SIMSD_ERR_ALIGNMENT, "attention: workspace must be 16-byte aligned");
    if (workspace_bytes < p.workspace)
      return fail(SIMSD_ERR_WORKSPACE, "attention: workspace smaller than simsd_verify_attention_workspace_size()");
  }
  return SIMSD_OK;
}

simsd_status plan_accept(const simsd_accept_desc* d, int cus, AcceptPlan* p, bool sampled) {
  if (!d || !p) return fail(SIMSD_ERR_NULL_POINTER, "accept: descriptor is NULL");
  if (cus < 1) return fail(SIMSD_ERR_HIP, "accept: the device reports no compute units");
  if (!known_dtype(d->logits_dtype))
    return fail(SIMSD_ERR_UNSUPPORTED, "accept: logits_dtype must be SIMSD_F32 or SIMSD_BF16");
  if (d->batch < 1 || d->batch > 65535)
    return fail(SIMSD_ERR_BAD_SHAPE, "accept: batch must be in [1, 65535]");
  if (d->block_size < 1 || d->block_size > kMaxNew)
    return fail(SIMSD_ERR_BAD_SHAPE, "accept: block_size must be in [1, 64]");
  if (d->max_ref < 0 || d->max_ref > d->block_size)
    return fail(SIMSD_ERR_BAD_SHAPE, "accept: need 0 <= max_ref <= block_size");
  if (d->vocab < 1) return fail(SIMSD_ERR_BAD_SHAPE, "accept: vocab must be >= 1");
  if (d->chunks_per_row < 0) return fail(SIMSD_ERR_BAD_SHAPE, "accept: chunks_per_row < 0");
  AcceptPlan r;
  r.rows = d->block_size + (sampled ? d->max_ref : 0);
  const int eb = elem_bytes(d->logits_dtype);
  const int w = 16 / eb;
  r.vec = (d->vocab % w == 0) ? w : 1;
  r.nvec = ceil_div(d->vocab, r.vec);
  const int64_t rows = static_cast<int64_t>(d->batch) * r.rows;
  int64_t cpr = d->chunks_per_row;
  if (cpr == 0) {
    cpr = ceil_div(int64_t{kAcceptPerCU} * cus, rows);
    const int64_t most = std::max<int64_t>(1, r.nvec / kAcceptThreads);
    if (cpr > most) cpr = most;
  }
  if (cpr > r.nvec) cpr = r.nvec;
  if (cpr > 65535 * 1024) return fail(SIMSD_ERR_BAD_SHAPE, "accept: chunks_per_row too large");
  r.cpr = static_cast<int>(cpr);
  r.chunk_vecs = ceil_div(r.nvec, r.cpr);
  r.workspace = static_cast<size_t>(rows) * r.cpr * sizeof(AcceptPartial);
  if (sampled) {
    // About kAcceptPerCU draw work-groups per compute unit, each at least one
    // vector per thread.
    int64_t g = ceil_div(int64_t{kAcceptPerCU} * cus, d->batch);
    const int64_t most = std::max<int64_t>(1, r.nvec / kAcceptThreads);
    g = std::min<int64_t>(std::min<int64_t>(g, most), kAcceptThreads);
    r.draw_chunks = static_cast<int>(std::max<int64_t>(g, 1));
    r.draw_vecs = ceil_div(r.nvec, r.draw_chunks);
    r.draw_row_off = (r.workspace + 255) / 256 * 256;
    r.draw_part_off = r.draw_row_off + static_cast<size_t>(d->batch) * sizeof(DrawRow);
    r.workspace = r.draw_part_off + static_cast<size_t>(d->batch) * r.draw_chunks * sizeof(DrawPartial);
  }
  *p = r;
  return SIMSD_OK;
}

simsd_status check_accept_inputs(const simsd_accept_desc* d, const void* logits,
                                 const int32_t* draft_ids, const int32_t* step_map,
                                 const int32_t* num_ref, const int32_t* target_ids,
                                 const int32_t* accept_len) {
  if (!logits || !step_map || !num_ref || !target_ids || !accept_len)
    return fail(SIMSD_ERR_NULL_POINTER,
                "accept: logits, step_map, num_ref, target_ids and accept_len are required");
  if (d->max_ref > 0 && !draft_ids)
    return fail(SIMSD_ERR_NULL_POINTER, "accept: draft_ids required when max_ref > 0");
  if (!aligned16(logits)) return fail(SIMSD_ERR_ALIGNMENT, "accept: logits must be 16-byte aligned");
  return SIMSD_OK;
}

simsd_status check_accept_args(const simsd_accept_desc* d, const AcceptPlan& p,
                               const void* logits, const int32_t* draft_ids,
                               const int32_t* step_map, const int32_t* num_ref,
                               const int32_t* target_ids, const float* confidence,
                               const float* draft_prob, const int32_t* accept_len,
                               const void* workspace, size_t workspace_bytes) {
  (void)confidence;
  (void)draft_prob;
  const simsd_status st = check_accept_inputs(d, logits, draft_ids, step_map, num_ref,
                                              target_ids, accept_len);
  if (st != SIMSD_OK) return st;
  if (!workspace) return fail(SIMSD_ERR_WORKSPACE, "accept: workspace is NULL");
  if (!aligned16(workspace)) return fail(SIMSD_ERR_ALIGNMENT, "accept: workspace must be 16-byte aligned");
  if (workspace_bytes < p.workspace)
    return fail(SIMSD_ERR_WORKSPACE, "accept: workspace smaller than simsd_verify_accept_workspace_size()");
  return SIMSD_OK;
}

simsd_status plan_lmhead(const simsd_lmhead_desc* d, int vocab_tile, int stage, LmheadPlan* p) {
  if (!d || !p) return fail(SIMSD_ERR_NULL_POINTER, "lmhead: descriptor is NULL");
  if (dtype_code(d->dtype) != SIMSD_BF16)
    return fail(SIMSD_ERR_UNSUPPORTED, "lmhead: dtype must be SIMSD_BF16");
  if (d->batch < 1 || d->batch > 65535)
    return fail(SIMSD_ERR_BAD_SHAPE, "lmhead: batch must be in [1, 65535]");
  if (d->block_size < 1 || d->block_size > kMaxNew)
    return fail(SIMSD_ERR_BAD_SHAPE, "lmhead: block_size must be in [1, 64]");
  if (d->max_ref < 0 || d->max_ref > d->block_size)
    return fail(SIMSD_ERR_BAD_SHAPE, "lmhead: need 0 <= max_ref <= block_size");
  if (d->vocab < 1) return fail(SIMSD_ERR_BAD_SHAPE, "lmhead: vocab must be >= 1");
  if (d->hidden < stage || d->hidden % stage != 0)
    return fail(SIMSD_ERR_BAD_SHAPE, "lmhead: hidden must be a positive multiple of 64");
  if (static_cast<int64_t>(d->batch) * d->block_size > (int64_t{1} << 24) ||
      static_cast<int64_t>(d->vocab) * d->hidden * 2 > (int64_t{1} << 40))
    return fail(SIMSD_ERR_BAD_SHAPE, "lmhead: sizes too large");
  LmheadPlan r;
  r.vtiles = static_cast<int>(ceil_div(d->vocab, vocab_tile));
  if (r.vtiles > 65535) return fail(SIMSD_ERR_BAD_SHAPE, "lmhead: vocab too large");
  // The scan's tile count (row tiles x vocabulary tiles) stays an int.
  if (static_cast<int64_t>(d->batch) * d->block_size * r.vtiles > (int64_t{1} << 30))
    return fail(SIMSD_ERR_BAD_SHAPE, "lmhead: batch * block_size * vocabulary tiles too large");
  const size_t parts = static_cast<size_t>(d->batch) * d->block_size * r.vtiles * sizeof(AcceptPartial);
  r.merged_off = (parts + 255) / 256 * 256;
  r.xdraft_off = (r.merged_off + static_cast<size_t>(d->batch) * d->block_size * sizeof(AcceptPartial) +
                  255) / 256 * 256;
  r.workspace = r.xdraft_off + static_cast<size_t>(d->batch) * std::max(d->max_ref, 1) * sizeof(float);
  *p = r;
  return SIMSD_OK;
}

simsd_status check_lmhead_args(const simsd_lmhead_desc* d, const LmheadPlan& p, const void* hidden,
                               const void* weight, const int32_t* draft_ids,
                               const int32_t* step_map, const int32_t* num_ref,
                               const int32_t* target_ids, const int32_t* accept_len,
                               const void* workspace, size_t workspace_bytes) {
  if (!hidden || !weight || !step_map || !num_ref || !target_ids || !accept_len)
    return fail(SIMSD_ERR_NULL_POINTER,
                "lmhead: hidden, weight, step_map, num_ref, target_ids and accept_len are required");
  if (d->max_ref > 0 && !draft_ids)
    return fail(SIMSD_ERR_NULL_POINTER, "lmhead: draft_ids required when max_ref > 0");
  if (!aligned16(hidden) || !aligned16(weight))
    return fail(SIMSD_ERR_ALIGNMENT, "lmhead: hidden and weight must be 16-byte aligned");
  if (!workspace) return fail(SIMSD_ERR_WORKSPACE, "lmhead: workspace is NULL");
  if (!aligned16(workspace)) return fail(SIMSD_ERR_ALIGNMENT, "lmhead: workspace must be 16-byte aligned");
  if (workspace_bytes < p.workspace)
    return fail(SIMSD_ERR_WORKSPACE,
                "lmhead: workspace smaller than simsd_verify_accept_lmhead_workspace_size()");
  return SIMSD_OK;
}

simsd_status check_accept_sampled_args(const simsd_accept_desc* d, const AcceptPlan& p,
                                       float temperature, const void* logits,
                                       const void* draft_logits, const int32_t* draft_ids,
                                       const int32_t* step_map, const int32_t* num_ref,
                                       const float* uniforms, const int32_t* accept_len,
                                       const int32_t* correction, const void* workspace,
                                       size_t workspace_bytes) {
  if (!(temperature > 0.f) || !std::isfinite(temperature))
    return fail(SIMSD_ERR_BAD_SHAPE, "accept_sampled: temperature must be finite and > 0");
  if (!logits || !step_map || !num_ref || !uniforms || !accept_len || !correction)
    return fail(SIMSD_ERR_NULL_POINTER,
                "accept_sampled: logits, step_map, num_ref, uniforms, accept_len and correction are required");
  if (d->max_ref > 0 && (!draft_ids || !draft_logits))
    return fail(SIMSD_ERR_NULL_POINTER,
                "accept_sampled: draft_ids and draft_logits required when max_ref > 0");
  if (!aligned16(logits) || (draft_logits && !aligned16(draft_logits)))
    return fail(SIMSD_ERR_ALIGNMENT, "accept_sampled: logits and draft_logits must be 16-byte aligned");
  if (!workspace) return fail(SIMSD_ERR_WORKSPACE, "accept_sampled: workspace is NULL");
  if (!aligned16(workspace))
    return fail(SIMSD_ERR_ALIGNMENT, "accept_sampled: workspace must be 16-byte aligned");
  if (workspace_bytes < p.workspace)
    return fail(SIMSD_ERR_WORKSPACE,
                "accept_sampled: workspace smaller than simsd_verify_accept_sampled_workspace_size()");
  return SIMSD_OK;
}

}  // namespace simsd

using namespace simsd;

extern "C" simsd_status simsd_validate_step_map(const int32_t* step_map, const int32_t* num_ref,
                                                int32_t batch, int32_t block_size,
                                                int32_t max_ref) {
  if (!step_map || !num_ref) return fail(SIMSD_ERR_NULL_POINTER, "validate_step_map: NULL array");
  if (batch < 1 || block_size < 1 || block_size > kMaxNew || max_ref < 0 || max_ref > block_size)
    return fail(SIMSD_ERR_BAD_SHAPE,
                "validate_step_map: need batch >= 1, 1 <= block_size <= 64, 0 <= max_ref <= block_size");
  int seen[kMaxNew + 1];
  for (int32_t b = 0; b < batch; ++b) {
    const int32_t gamma = num_ref[b];
    if (gamma < 0 || gamma > max_ref) {
      char buf[160];
      std::snprintf(buf, sizeof buf, "sequence %d: num_ref %d outside [0, %d]", b, gamma, max_ref);
      return fail(SIMSD_ERR_INVALID_STEP_MAP, buf);
    }
    std::fill(seen, seen + block_size + 1, 0);
    for (int32_t k = 0; k < block_size; ++k) {
      const int32_t s = step_map[static_cast<int64_t>(b) * block_size + k];
      if (s >= 1 && s <= gamma) ++seen[s];
    }
    for (int32_t r = 1; r <= gamma; ++r) {
      if (seen[r] != 1) {
        char buf[160];
        std::snprintf(buf, sizeof buf, "sequence %d: draft step %d occurs %d times (must be once)",
                      b, r, seen[r]);
        return fail(SIMSD_ERR_INVALID_STEP_MAP, buf);
      }
    }
  }
  return SIMSD_OK;
}

extern "C" const char* simsd_status_string(simsd_status s) {
  switch (s) {
    case SIMSD_OK: return "SIMSD_OK";
    case SIMSD_ERR_NULL_POINTER: return "SIMSD_ERR_NULL_POINTER";
    case SIMSD_ERR_BAD_SHAPE: return "SIMSD_ERR_BAD_SHAPE";
    case SIMSD_ERR_UNSUPPORTED: return "SIMSD_ERR_UNSUPPORTED";
    case SIMSD_ERR_ALIGNMENT: return "SIMSD_ERR_ALIGNMENT";
    case SIMSD_ERR_WORKSPACE: return "SIMSD_ERR_WORKSPACE";
    case SIMSD_ERR_INVALID_STEP_MAP: return "SIMSD_ERR_INVALID_STEP_MAP";
    case SIMSD_ERR_HIP: return "SIMSD_ERR_HIP";
  }
  return "SIMSD_ERR_UNKNOWN";
}

extern "C" const char* simsd_last_error(void) { return g_last_error.c_str(); }

extern "C" int simsd_version(void) { return SIMSD_VERSION; }
