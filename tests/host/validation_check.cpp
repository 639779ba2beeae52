// Host-only check of the C ABI's argument validation and launch planning.
//
// Built from simsd_plan.cpp alone (no HIP, no GPU) with g++ under
// -fsanitize=address,undefined by tests/test_host_sanitize.py: the planners
// and checkers of every entry point, the host helpers and the thread-local
// error string run through the error cases the Python ABI tests use, the
// workspace sizes of the workloads, and a seeded fuzz of descriptors with
// extreme values (which must be rejected or planned without undefined
// behaviour).  Pointers are small aligned fakes that are never dereferenced.
// Exit status 0 when every expectation holds; a sanitizer report aborts.
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <limits>
#include <random>
#include <string>

#include "simsd.h"
#include "simsd_plan.h"

using namespace simsd;

static int g_fail = 0;
static int g_checks = 0;

#define EXPECT(cond)                                                          \
  do {                                                                        \
    ++g_checks;                                                               \
    if (!(cond)) {                                                            \
      std::fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__,       \
                   __LINE__, #cond);                                          \
      ++g_fail;                                                               \
    }                                                                         \
  } while (0)

static const void* const FAKE = reinterpret_cast<const void*>(uintptr_t{0x10000});
static void* const FAKEW = reinterpret_cast<void*>(uintptr_t{0x10000});
static const int32_t* const FAKEI = reinterpret_cast<const int32_t*>(uintptr_t{0x10000});
static int32_t* const FAKEIW = reinterpret_cast<int32_t*>(uintptr_t{0x10000});
static constexpr int kCUs = 256;   // an MI355X

// The workloads: 1 tiny fp32, 2 SDAR-1.7B layer, 3 SDAR-8B layer,
// 4 long context, 5 ragged paged.
static simsd_attn_desc cfg_desc(int cid) {
  simsd_attn_desc d{};
  d.head_dim = cid == 1 ? 64 : 128;
  d.dtype = cid == 1 ? SIMSD_F32 : SIMSD_BF16;
  switch (cid) {
    case 1: d.batch = 1; d.num_q_heads = 2; d.num_kv_heads = 1; d.block_size = 4; d.max_ref = 4; d.max_prefix_len = 64; break;
    case 2: d.batch = 1; d.num_q_heads = 16; d.num_kv_heads = 8; d.block_size = 4; d.max_ref = 4; d.max_prefix_len = 1024; break;
    case 3: d.batch = 8; d.num_q_heads = 32; d.num_kv_heads = 8; d.block_size = 16; d.max_ref = 16; d.max_prefix_len = 4096; break;
    case 4: d.batch = 16; d.num_q_heads = 32; d.num_kv_heads = 8; d.block_size = 32; d.max_ref = 32; d.max_prefix_len = 16384; break;
    default: d.batch = 64; d.num_q_heads = 32; d.num_kv_heads = 8; d.block_size = 8; d.max_ref = 8; d.max_prefix_len = 32768; d.page_size = 16; break;
  }
  const int64_t hd = int64_t{d.num_kv_heads} * d.head_dim;
  if (d.page_size > 0) {
    d.max_pages_per_seq = (d.max_prefix_len + d.page_size - 1) / d.page_size;
    d.cache_stride_seq = d.page_size * hd;
  } else {
    d.cache_stride_seq = d.max_prefix_len * hd;
  }
  d.cache_stride_token = hd;
  d.cache_stride_head = d.head_dim;
  return d;
}

static simsd_status attn(const simsd_attn_desc& d, size_t ws_bytes = size_t{1} << 40,
                         const void* q = FAKE, const void* k_cache = FAKE,
                         const int32_t* block_table = FAKEI, const void* out = FAKE,
                         const float* lse = nullptr, const void* ws = FAKE, int cus = kCUs) {
  AttnPlan p;
  simsd_status st = plan_attention(&d, cus, &p);
  if (st != SIMSD_OK) return st;
  return check_attention_args(&d, p, q, FAKE, FAKE, k_cache, FAKE, block_table, FAKEI, FAKEI,
                              FAKEI, out, lse, ws, ws_bytes);
}

static size_t attn_ws(const simsd_attn_desc& d, int cus = kCUs) {
  AttnPlan p;
  return plan_attention(&d, cus, &p) == SIMSD_OK ? p.workspace : 0;
}

static bool last_error_set() { return std::strlen(simsd_last_error()) > 0; }

// Store an arbitrary integer in a dtype field, as a C caller can (forming an
// out-of-range enum value in C++ would itself be undefined).
static void set_dtype(simsd_dtype& field, int v) { std::memcpy(&field, &v, sizeof v); }

static void attention_cases() {
  // workspace sizes (the Python ABI tests check the same numbers)
  EXPECT(attn_ws(cfg_desc(4)) == size_t{128} * 2 * 256 * 130 * 4);
  simsd_attn_desc d = cfg_desc(4);
  d.kv_chunk = 4096;
  EXPECT(attn_ws(d) == size_t{128} * 4 * 256 * 130 * 4);
  d = cfg_desc(1);
  d.kv_chunk = 64;
  EXPECT(attn_ws(d) == 0);
  EXPECT(attn_ws(cfg_desc(2)) > 0);
  d = cfg_desc(2);
  d.kv_chunk = -1;
  EXPECT(attn_ws(d) == size_t{256} * 2 * 128 * 130 * 4 + 257 * 8);
  // fewer compute units: fewer resident groups, a smaller workspace
  EXPECT(attn_ws(d, 64) == size_t{64} * 2 * 128 * 130 * 4 + 257 * 8);
  EXPECT(attn_ws(cfg_desc(5)) > 0);
  EXPECT(attn(cfg_desc(5)) == SIMSD_OK);

  struct Case { const char* what; int status; void (*mut)(simsd_attn_desc&); };
  const Case cases[] = {
      {"head_dim 96", SIMSD_ERR_UNSUPPORTED, [](simsd_attn_desc& x) { x.head_dim = 96; }},
      {"head_dim 256", SIMSD_ERR_UNSUPPORTED, [](simsd_attn_desc& x) { x.head_dim = 256; }},
      {"Hq % Hkv", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.num_q_heads = 6; }},
      {"Hkv 0", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.num_kv_heads = 0; }},
      {"group 17", SIMSD_ERR_UNSUPPORTED, [](simsd_attn_desc& x) { x.num_q_heads = 136; }},
      {"B 0", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.block_size = 0; }},
      {"L > B", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.max_ref = 5; }},
      {"B + L > 64", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.block_size = 40; x.max_ref = 30; }},
      {"batch 0", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.batch = 0; }},
      {"batch 70000", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.batch = 70000; }},
      {"prefix -1", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.max_prefix_len = -1; }},
      {"chunk 100", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.kv_chunk = 100; }},
      {"chunk -64", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.kv_chunk = -64; }},
      {"chunk -2", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.kv_chunk = -2; }},
      {"page -2", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.page_size = -2; }},
      {"stream f32", SIMSD_ERR_UNSUPPORTED, [](simsd_attn_desc& x) { x.kv_chunk = -1; x.dtype = SIMSD_F32; }},
      {"stream batch", SIMSD_ERR_UNSUPPORTED, [](simsd_attn_desc& x) { x.kv_chunk = -1; x.batch = 257; }},
      {"stride 12", SIMSD_ERR_ALIGNMENT, [](simsd_attn_desc& x) { x.cache_stride_token = 12; }},
      {"stride -8", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.cache_stride_head = -8; }},
      {"stride huge", SIMSD_ERR_BAD_SHAPE,
       [](simsd_attn_desc& x) { x.cache_stride_seq = std::numeric_limits<int64_t>::max() - 7; }},
      {"scale -1", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.scale = -1.f; }},
      {"scale inf", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.scale = INFINITY; }},
      {"dtype 7", SIMSD_ERR_UNSUPPORTED, [](simsd_attn_desc& x) { set_dtype(x.dtype, 7); }},
      {"rope -1", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.rope_theta = -1.f; }},
      {"rope nan", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.rope_theta = NAN; }},
      {"rope inf", SIMSD_ERR_BAD_SHAPE, [](simsd_attn_desc& x) { x.rope_theta = INFINITY; }},
  };
  for (const Case& c : cases) {
    simsd_attn_desc x = cfg_desc(2);
    c.mut(x);
    const simsd_status st = attn(x);
    if (st != c.status) std::fprintf(stderr, "attention case %s: status %d\n", c.what, st);
    EXPECT(st == c.status);
    EXPECT(last_error_set());
  }
  simsd_attn_desc x = cfg_desc(4);
  x.kv_chunk = -1;                                  // 256 packed rows: no stream decomposition
  EXPECT(attn(x) == SIMSD_ERR_UNSUPPORTED);

  // pointers, alignment, workspace
  simsd_attn_desc w = cfg_desc(2);
  w.kv_chunk = 64;
  const size_t ws = attn_ws(w);
  EXPECT(ws > 0);
  EXPECT(attn(w, ws) == SIMSD_OK);
  EXPECT(attn(w, ws, nullptr) == SIMSD_ERR_NULL_POINTER);
  EXPECT(attn(w, ws, FAKE, nullptr) == SIMSD_ERR_NULL_POINTER);
  EXPECT(attn(w, ws, FAKE, FAKE, FAKEI, reinterpret_cast<const void*>(uintptr_t{0x10008})) ==
         SIMSD_ERR_ALIGNMENT);
  EXPECT(attn(w, ws, FAKE, FAKE, FAKEI, FAKE, reinterpret_cast<const float*>(uintptr_t{0x10002})) ==
         SIMSD_ERR_ALIGNMENT);
  EXPECT(attn(w, 0, FAKE, FAKE, FAKEI, FAKE, nullptr, nullptr) == SIMSD_ERR_WORKSPACE);
  EXPECT(attn(w, ws - 1) == SIMSD_ERR_WORKSPACE);
  EXPECT(attn(w, ws, FAKE, FAKE, FAKEI, FAKE, nullptr, FAKE, 0) == SIMSD_ERR_HIP);   // no units
  simsd_attn_desc pg = cfg_desc(5);
  EXPECT(attn(pg, size_t{1} << 40, FAKE, FAKE, nullptr) == SIMSD_ERR_NULL_POINTER);
  pg.max_pages_per_seq = 3;
  EXPECT(attn(pg) == SIMSD_ERR_BAD_SHAPE);
  // a zero-length prefix needs no cache
  simsd_attn_desc z = cfg_desc(2);
  z.max_prefix_len = 0;
  EXPECT(attn(z, 0, FAKE, nullptr, nullptr, FAKE, nullptr, nullptr) == SIMSD_OK);
}

static simsd_status accept_call(const simsd_accept_desc& d, size_t ws_bytes = size_t{1} << 30,
                                const void* logits = FAKE, const int32_t* draft = FAKEI,
                                const void* ws = FAKE) {
  AcceptPlan p;
  simsd_status st = plan_accept(&d, kCUs, &p);
  if (st != SIMSD_OK) return st;
  return check_accept_args(&d, p, logits, draft, FAKEI, FAKEI, FAKEIW, nullptr, nullptr, FAKEIW,
                           ws, ws_bytes);
}

static void accept_cases() {
  const simsd_accept_desc good{2, 4, 4, 1000, 0, SIMSD_BF16};
  EXPECT(accept_call(good) == SIMSD_OK);
  simsd_accept_desc big{16, 32, 32, 151936, 0, SIMSD_BF16};
  AcceptPlan p;
  EXPECT(plan_accept(&big, kCUs, &p) == SIMSD_OK && p.workspace == size_t{512} * 16);
  EXPECT(plan_accept(&big, kCUs, &p, true) == SIMSD_OK &&
         p.workspace == size_t{16} * 64 * 16 + 16 * 32 + 16 * 32 * 16);
  struct Case { int status; void (*mut)(simsd_accept_desc&); };
  const Case cases[] = {
      {SIMSD_ERR_BAD_SHAPE, [](simsd_accept_desc& x) { x.batch = 0; }},
      {SIMSD_ERR_BAD_SHAPE, [](simsd_accept_desc& x) { x.block_size = 65; }},
      {SIMSD_ERR_BAD_SHAPE, [](simsd_accept_desc& x) { x.max_ref = 5; }},
      {SIMSD_ERR_BAD_SHAPE, [](simsd_accept_desc& x) { x.vocab = 0; }},
      {SIMSD_ERR_BAD_SHAPE, [](simsd_accept_desc& x) { x.chunks_per_row = -1; }},
      {SIMSD_ERR_UNSUPPORTED, [](simsd_accept_desc& x) { set_dtype(x.logits_dtype, 3); }},
  };
  for (const Case& c : cases) {
    simsd_accept_desc x = good;
    c.mut(x);
    EXPECT(accept_call(x) == c.status);
  }
  EXPECT(accept_call(good, size_t{1} << 30, nullptr) == SIMSD_ERR_NULL_POINTER);
  EXPECT(accept_call(good, size_t{1} << 30, FAKE, nullptr) == SIMSD_ERR_NULL_POINTER);
  EXPECT(accept_call(good, size_t{1} << 30, reinterpret_cast<const void*>(uintptr_t{0x10004})) ==
         SIMSD_ERR_ALIGNMENT);
  EXPECT(accept_call(good, size_t{1} << 30, FAKE, FAKEI, nullptr) == SIMSD_ERR_WORKSPACE);
  EXPECT(plan_accept(&good, kCUs, &p) == SIMSD_OK);
  EXPECT(accept_call(good, p.workspace - 1) == SIMSD_ERR_WORKSPACE);

  // the stochastic rule
  EXPECT(plan_accept(&good, kCUs, &p, true) == SIMSD_OK);
  for (float t : {0.f, -1.f, INFINITY, NAN})
    EXPECT(check_accept_sampled_args(&good, p, t, FAKE, FAKE, FAKEI, FAKEI, FAKEI,
                                     reinterpret_cast<const float*>(FAKE), FAKEIW, FAKEIW, FAKE,
                                     p.workspace) == SIMSD_ERR_BAD_SHAPE);
  EXPECT(check_accept_sampled_args(&good, p, 1.f, FAKE, reinterpret_cast<const void*>(uintptr_t{0x10008}),
                                   FAKEI, FAKEI, FAKEI, reinterpret_cast<const float*>(FAKE), FAKEIW,
                                   FAKEIW, FAKE, p.workspace) == SIMSD_ERR_ALIGNMENT);
  EXPECT(check_accept_sampled_args(&good, p, 1.f, FAKE, FAKE, FAKEI, FAKEI, FAKEI, nullptr, FAKEIW,
                                   FAKEIW, FAKE, p.workspace) == SIMSD_ERR_NULL_POINTER);
  EXPECT(check_accept_sampled_args(&good, p, 1.f, FAKE, FAKE, FAKEI, FAKEI, FAKEI,
                                   reinterpret_cast<const float*>(FAKE), FAKEIW, FAKEIW, FAKE,
                                   p.workspace - 1) == SIMSD_ERR_WORKSPACE);
}

static void lmhead_cases() {
  const simsd_lmhead_desc good{2, 4, 4, 1000, 128, SIMSD_BF16};
  LmheadPlan p;
  EXPECT(plan_lmhead(&good, 128, 64, &p) == SIMSD_OK);
  const size_t R = 8, vt = (1000 + 127) / 128;
  const size_t merged = (R * vt * 16 + 255) / 256 * 256;
  const size_t xdraft = (merged + R * 16 + 255) / 256 * 256;
  EXPECT(p.workspace == xdraft + 2 * 4 * 4);
  struct Case { int status; void (*mut)(simsd_lmhead_desc&); };
  const Case cases[] = {
      {SIMSD_ERR_BAD_SHAPE, [](simsd_lmhead_desc& x) { x.batch = 0; }},
      {SIMSD_ERR_BAD_SHAPE, [](simsd_lmhead_desc& x) { x.block_size = 65; }},
      {SIMSD_ERR_BAD_SHAPE, [](simsd_lmhead_desc& x) { x.max_ref = 5; }},
      {SIMSD_ERR_BAD_SHAPE, [](simsd_lmhead_desc& x) { x.vocab = 0; }},
      {SIMSD_ERR_BAD_SHAPE, [](simsd_lmhead_desc& x) { x.hidden = 0; }},
      {SIMSD_ERR_BAD_SHAPE, [](simsd_lmhead_desc& x) { x.hidden = 96; }},
      {SIMSD_ERR_UNSUPPORTED, [](simsd_lmhead_desc& x) { x.dtype = SIMSD_F32; }},
      {SIMSD_ERR_BAD_SHAPE, [](simsd_lmhead_desc& x) { x.vocab = std::numeric_limits<int32_t>::max(); }},
  };
  for (const Case& c : cases) {
    simsd_lmhead_desc x = good;
    c.mut(x);
    EXPECT(plan_lmhead(&x, 128, 64, &p) == c.status);
  }
  EXPECT(plan_lmhead(&good, 128, 64, &p) == SIMSD_OK);
  EXPECT(check_lmhead_args(&good, p, nullptr, FAKE, FAKEI, FAKEI, FAKEI, FAKEIW, FAKEIW, FAKE,
                           p.workspace) == SIMSD_ERR_NULL_POINTER);
  EXPECT(check_lmhead_args(&good, p, reinterpret_cast<const void*>(uintptr_t{0x10008}), FAKE, FAKEI,
                           FAKEI, FAKEI, FAKEIW, FAKEIW, FAKE, p.workspace) == SIMSD_ERR_ALIGNMENT);
  EXPECT(check_lmhead_args(&good, p, FAKE, FAKE, FAKEI, FAKEI, FAKEI, FAKEIW, FAKEIW, FAKE,
                           p.workspace - 1) == SIMSD_ERR_WORKSPACE);
  EXPECT(check_lmhead_args(&good, p, FAKE, FAKE, FAKEI, FAKEI, FAKEI, FAKEIW, FAKEIW, FAKE,
                           p.workspace) == SIMSD_OK);
}

static void host_helper_cases() {
  const int32_t ok[] = {2, 1, 0, -1, 9, 1, 2, 3, 4, 5};
  const int32_t ok_g[] = {2, 5};
  EXPECT(simsd_validate_step_map(ok, ok_g, 2, 5, 5) == SIMSD_OK);
  const int32_t dup[] = {1, 1, 0, 0, 0};
  const int32_t two[] = {2};
  EXPECT(simsd_validate_step_map(dup, two, 1, 5, 5) == SIMSD_ERR_INVALID_STEP_MAP);
  const int32_t gap[] = {2, 3, 0, 0, 0};
  EXPECT(simsd_validate_step_map(gap, two, 1, 5, 5) == SIMSD_ERR_INVALID_STEP_MAP);
  const int32_t six[] = {6}, neg[] = {-1};
  const int32_t m12[] = {1, 2, 0, 0, 0};
  EXPECT(simsd_validate_step_map(m12, six, 1, 5, 5) == SIMSD_ERR_INVALID_STEP_MAP);
  EXPECT(simsd_validate_step_map(m12, neg, 1, 5, 5) == SIMSD_ERR_INVALID_STEP_MAP);
  EXPECT(std::strstr(simsd_last_error(), "sequence 0") != nullptr);
  EXPECT(simsd_validate_step_map(nullptr, two, 1, 5, 5) == SIMSD_ERR_NULL_POINTER);
  EXPECT(simsd_validate_step_map(m12, two, 1, 65, 5) == SIMSD_ERR_BAD_SHAPE);
  EXPECT(simsd_validate_step_map(m12, two, 1, std::numeric_limits<int32_t>::max(), 5) ==
         SIMSD_ERR_BAD_SHAPE);
  EXPECT(simsd_validate_step_map(m12, two, 0, 5, 5) == SIMSD_ERR_BAD_SHAPE);
  for (int c = 0; c <= 7; ++c)
    EXPECT(std::strncmp(simsd_status_string(static_cast<simsd_status>(c)), "SIMSD_", 6) == 0);
  EXPECT(std::strcmp(simsd_status_string(static_cast<simsd_status>(99)), "SIMSD_ERR_UNKNOWN") == 0);
  EXPECT(simsd_version() == SIMSD_VERSION);
}

// Seeded fuzz: descriptors drawn from small, typical and extreme values.  The
// planners must reject them or produce a plan whose sizes are consistent,
// without undefined behaviour (the sanitizers abort on any).
static int32_t pick32(std::mt19937_64& g) {
  static const int32_t edge[] = {0, 1, -1, 2, 3, 4, 7, 8, 15, 16, 17, 31, 32, 33, 63, 64, 65,
                                 96, 127, 128, 255, 256, 1000, 4096, 16384, 32768, 65535, 65536,
                                 151936, 1 << 24, std::numeric_limits<int32_t>::max(),
                                 std::numeric_limits<int32_t>::min()};
  if (g() % 4 == 0) return static_cast<int32_t>(g());
  return edge[g() % (sizeof edge / sizeof edge[0])];
}

static int64_t pick64(std::mt19937_64& g) {
  static const int64_t edge[] = {0, 8, 16, 64, 128, 1024, 1 << 20, int64_t{1} << 40,
                                 int64_t{1} << 48, (int64_t{1} << 48) + 8, -8,
                                 std::numeric_limits<int64_t>::max() - 7,
                                 std::numeric_limits<int64_t>::min()};
  if (g() % 4 == 0) return static_cast<int64_t>(g());
  return edge[g() % (sizeof edge / sizeof edge[0])];
}

static float pickf(std::mt19937_64& g) {
  static const float edge[] = {0.f, 1.f, 0.125f, -1.f, 1e4f, 1e38f, INFINITY, -INFINITY, NAN};
  return edge[g() % (sizeof edge / sizeof edge[0])];
}

static void fuzz(int iters) {
  std::mt19937_64 g(20241202);
  int planned = 0;
  for (int i = 0; i < iters; ++i) {
    simsd_attn_desc d{};
    d.batch = pick32(g);
    d.num_q_heads = pick32(g);
    d.num_kv_heads = pick32(g);
    d.head_dim = (g() % 2) ? ((g() % 2) ? 64 : 128) : pick32(g);
    d.block_size = pick32(g);
    d.max_ref = pick32(g);
    d.max_prefix_len = pick32(g);
    d.page_size = (g() % 2) ? 0 : pick32(g);
    d.max_pages_per_seq = pick32(g);
    d.kv_chunk = (g() % 3) ? 0 : pick32(g);
    d.cache_stride_seq = pick64(g);
    d.cache_stride_token = pick64(g);
    d.cache_stride_head = pick64(g);
    d.scale = pickf(g);
    d.rope_theta = pickf(g);
    set_dtype(d.dtype, static_cast<int>(g() % 3) - (g() % 7 == 0 ? 1000 : 0));
    const int cus = (g() % 2) ? 256 : static_cast<int>(g() % 1100) - 50;
    AttnPlan p;
    if (plan_attention(&d, cus, &p) == SIMSD_OK) {
      ++planned;
      EXPECT(p.splits >= 1 && p.rows_pb >= 1 && p.row_blocks >= 1 && p.chunk >= kTile);
      EXPECT(!p.stream || p.stream_groups >= 1);
      (void)check_attention_args(&d, p, FAKE, FAKE, FAKE, FAKE, FAKE, FAKEI, FAKEI, FAKEI, FAKEI,
                                 FAKE, nullptr, FAKE, p.workspace);
    }
    simsd_accept_desc a{pick32(g), pick32(g), pick32(g), pick32(g), (g() % 2) ? 0 : pick32(g),
                        SIMSD_F32};
    set_dtype(a.logits_dtype, static_cast<int>(g() % 3));
    AcceptPlan ap;
    if (plan_accept(&a, cus, &ap, g() % 2) == SIMSD_OK) {
      ++planned;
      EXPECT(ap.cpr >= 1 && ap.chunk_vecs >= 1 && ap.cpr * ap.chunk_vecs >= ap.nvec);
    }
    simsd_lmhead_desc l{pick32(g), pick32(g), pick32(g), pick32(g), pick32(g), SIMSD_BF16};
    set_dtype(l.dtype, static_cast<int>(g() % 3));
    LmheadPlan lp;
    if (plan_lmhead(&l, (g() % 2) ? 128 : 256, 64, &lp) == SIMSD_OK) {
      ++planned;
      EXPECT(lp.vtiles >= 1 && lp.workspace > lp.xdraft_off && lp.xdraft_off > lp.merged_off);
    }
    int32_t sm[64 * 4], nr[4];
    for (int& x : sm) x = static_cast<int32_t>(g() % 70) - 3;
    for (int& x : nr) x = static_cast<int32_t>(g() % 70) - 3;
    const int32_t B = static_cast<int32_t>(g() % 66), L = static_cast<int32_t>(g() % 66) - 1;
    const int32_t bt = static_cast<int32_t>(g() % 5);
    if (B <= 64) (void)simsd_validate_step_map(sm, nr, bt, B, L);
  }
  std::printf("fuzz: %d descriptors, %d planned\n", 3 * iters, planned);
}

int main() {
  attention_cases();
  accept_cases();
  lmhead_cases();
  host_helper_cases();
  fuzz(200000);
  std::printf("%d checks, %d failed\n", g_checks, g_fail);
  return g_fail == 0 ? 0 : 1;
}
