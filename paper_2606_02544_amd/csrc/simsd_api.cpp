// extern "C" compute entry points: check, plan, fill the argument block, launch.
#include <hip/hip_runtime.h>

#include <atomic>
#include <string>

#include "simsd.h"
#include "simsd_kernels.h"
#include "simsd_plan.h"

using namespace simsd;

static constexpr float kLog2eHost = 1.4426950408889634f;  // log2(e)

static simsd_status hip_fail(hipError_t e, const char* what) {
  set_error(std::string(what) + ": " + hipGetErrorString(e));
  return SIMSD_ERR_HIP;
}

// Compute units of device `dev`, queried once per device and cached (an
// attribute query: no allocation, no synchronisation).  A compute-partitioned
// MI355X reports the units of its partition.
static constexpr int kMaxDevices = 64;
static std::atomic<int> g_device_cus[kMaxDevices];

static hipError_t device_cus(int dev, int* cus) {
  if (dev >= 0 && dev < kMaxDevices) {
    const int v = g_device_cus[dev].load(std::memory_order_relaxed);
    if (v > 0) {
      *cus = v;
      return hipSuccess;
    }
  }
  int n = 0;
  const hipError_t e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  if (n < 1) return hipErrorInvalidDevice;
  if (dev >= 0 && dev < kMaxDevices) g_device_cus[dev].store(n, std::memory_order_relaxed);
  *cus = n;
  return hipSuccess;
}

// Device and compute units of the device a stream belongs to (the current
// device for the null stream).  When the query fails, *cus is the nominal
// count of an MI355X, so that argument errors are still reported first; the
// caller returns the query's error after validation.
static constexpr int kNominalCUs = 256;

hipError_t simsd::stream_device(void* stream, int* dev, int* cus) {
  hipDevice_t d = 0;
  hipError_t e = hipStreamGetDevice(static_cast<hipStream_t>(stream), &d);
  if (e == hipSuccess) e = device_cus(d, cus);
  if (e != hipSuccess) *cus = kNominalCUs;
  *dev = d;
  return e;
}

static hipError_t stream_cus(void* stream, int* cus) {
  int dev = 0;
  return stream_device(stream, &dev, cus);
}

// Compute units of the current device (workspace-size queries have no
// stream); the nominal count when no device is visible.
static int current_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || device_cus(dev, &cus) != hipSuccess) return kNominalCUs;
  return cus;
}

extern "C" size_t simsd_verify_attention_workspace_size(const simsd_attn_desc* desc) {
  AttnPlan p;
  if (plan_attention(desc, current_cus(), &p) != SIMSD_OK) return 0;
  return p.workspace;
}

extern "C" size_t simsd_verify_accept_workspace_size(const simsd_accept_desc* desc) {
  AcceptPlan p;
  if (plan_accept(desc, current_cus(), &p) != SIMSD_OK) return 0;
  return p.workspace;
}

extern "C" size_t simsd_verify_accept_sampled_workspace_size(const simsd_accept_desc* desc) {
  AcceptPlan p;
  if (plan_accept(desc, current_cus(), &p, true) != SIMSD_OK) return 0;
  return p.workspace;
}

extern "C" simsd_status simsd_verify_attention(
    const simsd_attn_desc* desc, const void* q, const void* k_new, const void* v_new,
    const void* k_cache, const void* v_cache, const int32_t* block_table,
    const int32_t* prefix_lens, const int32_t* step_map, const int32_t* num_ref, void* out,
    float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  try {
    int cus = 0;
    const hipError_t qe = stream_cus(stream, &cus);
    AttnPlan p;
    simsd_status st = plan_attention(desc, cus, &p);
    if (st != SIMSD_OK) return st;
    st = check_attention_args(desc, p, q, k_new, v_new, k_cache, v_cache, block_table,
                              prefix_lens, step_map, num_ref, out, lse, workspace,
                              workspace_bytes);
    if (st != SIMSD_OK) return st;
    if (qe != hipSuccess) return hip_fail(qe, "simsd_verify_attention: device query");
    AttnArgs a{};
    a.q = q;
    a.k_new = k_new;
    a.v_new = v_new;
    a.k_cache = k_cache;
    a.v_cache = v_cache;
    a.block_table = desc->page_size > 0 ? block_table : nullptr;
    a.prefix_lens = prefix_lens;
    a.step_map = step_map;
    a.num_ref = num_ref;
    a.out = out;
    a.lse = lse;
    a.part = p.workspace ? static_cast<float*>(workspace) : nullptr;
    a.stream_groups = p.stream ? p.stream_groups : 0;
    a.stream_seq0 = p.stream ? reinterpret_cast<int64_t*>(static_cast<char*>(workspace) +
                                                          static_cast<size_t>(p.stream_groups) * 2 *
                                                              p.part_floats * 4)
                             : nullptr;
    a.batch = desc->batch;
    a.cs_seq = desc->cache_stride_seq;
    a.cs_tok = desc->cache_stride_token;
    a.cs_head = desc->cache_stride_head;
    a.hq = desc->num_q_heads;
    a.hkv = desc->num_kv_heads;
    a.group = p.group;
    a.B = desc->block_size;
    a.L = desc->max_ref;
    a.n_new = p.n_new;
    a.rows = p.rows;
    a.rows_pb = p.rows_pb;
    a.row_blocks = p.row_blocks;
    a.page_size = desc->page_size > 0 ? desc->page_size : 1;
    a.max_pages = desc->max_pages_per_seq;
    a.chunk = p.chunk;
    a.splits = p.splits;
    a.max_prefix = desc->max_prefix_len;
    a.scale_log2 = p.scale_log2;
    a.rope = desc->rope_theta > 0.f ? 1 : 0;
    a.rope_step = p.rope_step;
    a.rope_theta = desc->rope_theta;
    const hipError_t e = launch_attention(*desc, p, a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "simsd_verify_attention launch");
    return SIMSD_OK;
  } catch (...) {
    set_error("simsd_verify_attention: internal error");
    return SIMSD_ERR_HIP;
  }
}

extern "C" simsd_status simsd_verify_accept(const simsd_accept_desc* desc, const void* logits,
                                            const int32_t* draft_ids, const int32_t* step_map,
                                            const int32_t* num_ref, int32_t* target_ids,
                                            float* confidence, float* draft_prob,
                                            int32_t* accept_len, void* workspace,
                                            size_t workspace_bytes, void* stream) {
  try {
    int cus = 0;
    const hipError_t qe = stream_cus(stream, &cus);
    AcceptPlan p;
    simsd_status st = plan_accept(desc, cus, &p);
    if (st != SIMSD_OK) return st;
    st = check_accept_args(desc, p, logits, draft_ids, step_map, num_ref, target_ids,
                           confidence, draft_prob, accept_len, workspace, workspace_bytes);
    if (st != SIMSD_OK) return st;
    if (qe != hipSuccess) return hip_fail(qe, "simsd_verify_accept: device query");
    AcceptArgs a{};
    a.logits = logits;
    a.draft_ids = draft_ids;
    a.step_map = step_map;
    a.num_ref = num_ref;
    a.target_ids = target_ids;
    a.confidence = confidence;
    a.draft_prob = draft_prob;
    a.accept_len = accept_len;
    a.part = static_cast<AcceptPartial*>(workspace);
    a.nvec = p.nvec;
    a.chunk_vecs = p.chunk_vecs;
    a.B = desc->block_size;
    a.L = desc->max_ref;
    a.V = desc->vocab;
    a.cpr = p.cpr;
    a.rows = p.rows;
    a.cl = kLog2eHost;
    const hipError_t e = launch_accept(*desc, p, a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "simsd_verify_accept launch");
    return SIMSD_OK;
  } catch (...) {
    set_error("simsd_verify_accept: internal error");
    return SIMSD_ERR_HIP;
  }
}

// Rows of the LM-head product, which pick the kernel variant and its vocabulary
// tile (0 for a NULL descriptor, which the plan then rejects).
static int lmhead_rows(const simsd_lmhead_desc* d) {
  if (!d) return 0;
  return static_cast<int>(std::min<int64_t>(int64_t{d->batch} * d->block_size, INT32_MAX));
}

extern "C" size_t simsd_verify_accept_lmhead_workspace_size(const simsd_lmhead_desc* desc) {
  LmheadPlan p;
  if (plan_lmhead(desc, lmhead_vocab_tile(lmhead_rows(desc)), lmhead_stage(), &p) != SIMSD_OK) return 0;
  return p.workspace;
}

extern "C" simsd_status simsd_verify_accept_lmhead(
    const simsd_lmhead_desc* desc, const void* hidden, const void* weight,
    const int32_t* draft_ids, const int32_t* step_map, const int32_t* num_ref,
    int32_t* target_ids, float* confidence, float* draft_prob, int32_t* accept_len,
    void* workspace, size_t workspace_bytes, void* stream) {
  try {
    LmheadPlan p;
    simsd_status st = plan_lmhead(desc, lmhead_vocab_tile(lmhead_rows(desc)), lmhead_stage(), &p);
    if (st != SIMSD_OK) return st;
    st = check_lmhead_args(desc, p, hidden, weight, draft_ids, step_map, num_ref, target_ids,
                           accept_len, workspace, workspace_bytes);
    if (st != SIMSD_OK) return st;
    float* xdraft = reinterpret_cast<float*>(static_cast<char*>(workspace) + p.xdraft_off);
    LmheadArgs l{};
    l.hidden = hidden;
    l.weight = weight;
    l.draft_ids = draft_ids;
    l.step_map = step_map;
    l.num_ref = num_ref;
    l.part = static_cast<AcceptPartial*>(workspace);
    l.merged = reinterpret_cast<AcceptPartial*>(static_cast<char*>(workspace) + p.merged_off);
    l.xdraft = xdraft;
    l.R = desc->batch * desc->block_size;
    l.B = desc->block_size;
    l.L = desc->max_ref;
    l.V = desc->vocab;
    l.H = desc->hidden;
    l.vtiles = p.vtiles;
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = launch_lmhead_scan(l, s);
    if (e == hipSuccess) e = launch_lmhead_merge(l, s);
    if (e != hipSuccess) return hip_fail(e, "simsd_verify_accept_lmhead launch");
    AcceptArgs a{};
    a.draft_ids = draft_ids;
    a.step_map = step_map;
    a.num_ref = num_ref;
    a.target_ids = target_ids;
    a.confidence = confidence;
    a.draft_prob = draft_prob;
    a.accept_len = accept_len;
    a.part = l.merged;
    a.B = desc->block_size;
    a.L = desc->max_ref;
    a.V = desc->vocab;
    a.cpr = 1;
    a.rows = desc->block_size;
    a.cl = kLog2eHost;
    a.xdraft = xdraft;
    e = launch_finalize_lmhead(desc->batch, a, s);
    if (e != hipSuccess) return hip_fail(e, "simsd_verify_accept_lmhead launch");
    return SIMSD_OK;
  } catch (...) {
    set_error("simsd_verify_accept_lmhead: internal error");
    return SIMSD_ERR_HIP;
  }
}

extern "C" simsd_status simsd_verify_accept_sampled(
    const simsd_accept_desc* desc, float temperature, const void* logits, const void* draft_logits,
    const int32_t* draft_ids, const int32_t* step_map, const int32_t* num_ref,
    const float* uniforms, float* p_target, float* p_draft, int32_t* accept_len,
    int32_t* correction, void* workspace, size_t workspace_bytes, void* stream) {
  try {
    int cus = 0;
    const hipError_t qe = stream_cus(stream, &cus);
    AcceptPlan p;
    simsd_status st = plan_accept(desc, cus, &p, true);
    if (st != SIMSD_OK) return st;
    st = check_accept_sampled_args(desc, p, temperature, logits, draft_logits, draft_ids, step_map,
                                   num_ref, uniforms, accept_len, correction, workspace,
                                   workspace_bytes);
    if (st != SIMSD_OK) return st;
    if (qe != hipSuccess) return hip_fail(qe, "simsd_verify_accept_sampled: device query");
    AcceptArgs a{};
    a.logits = logits;
    a.draft_logits = draft_logits;
    a.draft_ids = draft_ids;
    a.step_map = step_map;
    a.num_ref = num_ref;
    a.uniforms = uniforms;
    a.draft_prob = p_target;
    a.p_draft = p_draft;
    a.accept_len = accept_len;
    a.correction = correction;
    a.part = static_cast<AcceptPartial*>(workspace);
    a.nvec = p.nvec;
    a.chunk_vecs = p.chunk_vecs;
    a.B = desc->block_size;
    a.L = desc->max_ref;
    a.V = desc->vocab;
    a.cpr = p.cpr;
    a.rows = p.rows;
    a.cl = kLog2eHost / temperature;
    a.draw_chunks = p.draw_chunks;
    a.draw_vecs = p.draw_vecs;
    a.draw_row = reinterpret_cast<DrawRow*>(static_cast<char*>(workspace) + p.draw_row_off);
    a.draw_part = reinterpret_cast<DrawPartial*>(static_cast<char*>(workspace) + p.draw_part_off);
    const hipError_t e = launch_accept_sampled(*desc, p, a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "simsd_verify_accept_sampled launch");
    return SIMSD_OK;
  } catch (...) {
    set_error("simsd_verify_accept_sampled: internal error");
    return SIMSD_ERR_HIP;
  }
}
