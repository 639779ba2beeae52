// Vocabulary scan and acceptance of SimSD on gfx950.
//
// Eq. 2 at temperature 0 (Sec. 3.2): draft r is accepted while the target's
// argmax at its verification slot equals it, and the longest such prefix is
// kept.  Each logits row of a scanned block slot (step_map >= 1) is split into
// chunks; one work-group streams a chunk with 16-byte loads and keeps, per
// lane, the running maximum, the first vector reaching it and the sum of
// exp(x - max).  Partials are merged in (value desc, index asc) order, so ties
// resolve to the lowest vocabulary index exactly.  A second kernel, one
// work-group per sequence, issues its loads in two rounds (step map, drafts
// and every chunk partial of its rows; then the drafted tokens' logits),
// merges the chunks, computes confidence and draft probabilities and finds the
// accepted prefix with one wave ballot.
//
// The stochastic form of eq. 2 (temperature T, caller-supplied uniforms) runs
// the same scan over the verification rows and the drafter's rows, then the
// acceptance test and the residual draw of the first rejection (see the
// section further down).
#include <atomic>
#include <mutex>
#include <string>

#include "simsd_kernels.h"

// Scratch of simsd_verify_accept_noalloc: the scan partials of one call, in a
// fixed device array instead of a caller workspace.  Every GPU the library
// runs on holds its own copy until the process ends.  In host code the name
// `scratch` is only a host-side stand-in: host code uses the device address
// that scratch_address() obtains for each device, never the name itself.
static __device__ __align__(256) unsigned char scratch[SIMSD_NOALLOC_SCRATCH_BYTES];

namespace simsd {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kNoIndex = 0x7fffffff;
constexpr int NT = kAcceptThreads;

struct Best {
  float mx;
  int ix;
  float sm;  // sum of exp(x - mx)
};

// cl = log2(e) / T: the sums are of exp((x - max) / T).
__device__ inline Best combine(Best a, Best b, float cl) {
  const float M = fmaxf(a.mx, b.mx);
  Best r;
  r.mx = M;
  r.ix = a.mx > b.mx ? a.ix : (b.mx > a.mx ? b.ix : min(a.ix, b.ix));
  const float sa = a.mx == kNegInf ? 0.f : a.sm * __builtin_amdgcn_exp2f((a.mx - M) * cl);
  const float sb = b.mx == kNegInf ? 0.f : b.sm * __builtin_amdgcn_exp2f((b.mx - M) * cl);
  r.sm = sa + sb;
  return r;
}

__device__ inline Best wave_reduce(Best v, float cl) {
#pragma unroll
  for (int sh = 32; sh >= 1; sh >>= 1) {
    Best o;
    o.mx = __shfl_xor(v.mx, sh);
    o.ix = __shfl_xor(v.ix, sh);
    o.sm = __shfl_xor(v.sm, sh);
    v = combine(v, o, cl);
  }
  return v;
}

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

template <bool BF16>
__device__ inline float load_elem(const void* row, int64_t i) {
  if constexpr (BF16)
    return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(row)[i]) << 16);
  else
    return static_cast<const float*>(row)[i];
}

// Values of vector v of a row (VEC elements).
template <bool BF16, int VEC>
__device__ inline void load_vec(const void* row, int64_t v, float (&x)[VEC]) {
  if constexpr (VEC == 8) {
    const u32x4 w = reinterpret_cast<const u32x4*>(row)[v];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      x[2 * i] = bf16_lo(w[i]);
      x[2 * i + 1] = bf16_hi(w[i]);
    }
  } else if constexpr (VEC == 4) {
    const f32x4 w = reinterpret_cast<const f32x4*>(row)[v];
#pragma unroll
    for (int i = 0; i < 4; ++i) x[i] = w[i];
  } else {
    x[0] = load_elem<BF16>(row, v);
  }
}

// Scan vectors [v0, v1) of one row; returns this work-group's (max, index, sum).
template <bool BF16, int VEC>
__device__ Best scan_chunk(const void* row, int64_t v0, int64_t v1, int tid, float cl, Best* s_red) {
  float mx = kNegInf, sm = 0.f;
  int64_t vbest = -1;
  constexpr int U = 4;
  int64_t v = v0 + tid;
  for (; v + (U - 1) * NT < v1; v += U * NT) {
    float x[U][VEC];
#pragma unroll
    for (int u = 0; u < U; ++u) load_vec<BF16, VEC>(row, v + u * NT, x[u]);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float vm = x[u][0];
#pragma unroll
      for (int i = 1; i < VEC; ++i) vm = fmaxf(vm, x[u][i]);
      if (vm > mx) {
        sm = mx == kNegInf ? 0.f : sm * __builtin_amdgcn_exp2f((mx - vm) * cl);
        mx = vm;
        vbest = v + u * NT;
      }
      const float off = mx * cl;
#pragma unroll
      for (int i = 0; i < VEC; ++i) sm += __builtin_amdgcn_exp2f(fmaf(x[u][i], cl, -off));
    }
  }
  for (; v < v1; v += NT) {
    float x[VEC];
    load_vec<BF16, VEC>(row, v, x);
    float vm = x[0];
#pragma unroll
    for (int i = 1; i < VEC; ++i) vm = fmaxf(vm, x[i]);
    if (vm > mx) {
      sm = mx == kNegInf ? 0.f : sm * __builtin_amdgcn_exp2f((mx - vm) * cl);
      mx = vm;
      vbest = v;
    }
    const float off = mx * cl;
#pragma unroll
    for (int i = 0; i < VEC; ++i) sm += __builtin_amdgcn_exp2f(fmaf(x[i], cl, -off));
  }
  Best me = {kNegInf, kNoIndex, 0.f};
  if (vbest >= 0) {
    float x[VEC];
    load_vec<BF16, VEC>(row, vbest, x);
    int first = VEC - 1;
#pragma unroll
    for (int i = VEC - 1; i >= 0; --i)
      if (x[i] == mx) first = i;
    me.mx = mx;
    me.ix = static_cast<int>(vbest * VEC + first);
    me.sm = sm;
  }
  me = wave_reduce(me, cl);
  const int lane = tid & 63, wave = tid >> 6;
  if (lane == 0) s_red[wave] = me;
  __syncthreads();
  Best r = s_red[0];
  for (int i = 1; i < NT / 64; ++i) r = combine(r, s_red[i], cl);
  return r;
}

// One work-group per (vocabulary chunk, block slot, sequence): writes the
// chunk's (max, lowest index, sum of exp) to the workspace.
// Greedy: row y < B is block slot y, scanned when its step is >= 1.  Sampled:
// rows y < B are the verification rows (steps 1..gamma), and row B + r is the
// drafter's logits for draft r + 1 (r < gamma).
template <bool BF16, int VEC, bool SAMPLED>
__global__ void __launch_bounds__(NT) scan_kernel(AcceptArgs a) {
  __shared__ Best s_red[NT / 64];
  const int c = blockIdx.x, y = blockIdx.y, b = blockIdx.z;
  const int esz = BF16 ? 2 : 4;
  const char* row;
  if (!SAMPLED || y < a.B) {                 // (greedy grids have B rows: no test)
    const int step = a.step_map[static_cast<int64_t>(b) * a.B + y];
    if (step < 1) return;                    // committed or padding: not scanned
    if (SAMPLED && step > min(max(a.num_ref[b], 0), a.L)) return;   // not drafted
    row = static_cast<const char*>(a.logits) + (static_cast<int64_t>(b) * a.B + y) * a.V * esz;
  } else {
    const int r = y - a.B;
    if (r >= min(max(a.num_ref[b], 0), a.L)) return;
    row = static_cast<const char*>(a.draft_logits) + (static_cast<int64_t>(b) * a.L + r) * a.V * esz;
  }
  const int64_t v0 = static_cast<int64_t>(c) * a.chunk_vecs;
  const int64_t v1 = min(a.nvec, v0 + a.chunk_vecs);
  const Best r = scan_chunk<BF16, VEC>(row, v0, v1, threadIdx.x, a.cl, s_red);
  if (threadIdx.x == 0) {
    AcceptPartial pr;
    pr.mx = r.mx;
    pr.ix = r.ix;
    pr.sm = r.sm;
    pr.pad = 0;
    a.part[(static_cast<int64_t>(b) * a.rows + y) * a.cpr + c] = pr;
  }
}

// Partials a wave keeps in registers when it loads all its rows at once.
constexpr int kFinalRegs = 16;

// Loads the chunk partials of this wave's rows (wave, wave + NWV, ... < nr),
// PPL per lane per row, all before the first wait; returns them in registers.
template <int PPL>
__device__ inline void load_rows(const AcceptArgs& a, const AcceptPartial* pb, int nr, int wave,
                                 int lane, AcceptPartial (&buf)[kFinalRegs]) {
  constexpr int NWV = NT / 64;
  // Indices are clamped so that every load is unconditional and in bounds
  // (a guarded load would make the compiler wait on it right away); the merge
  // ignores the duplicates.
#pragma unroll
  for (int i = 0; i < kFinalRegs; ++i) {
    const int kk = min(wave + NWV * (i / PPL), nr - 1), cc = min(lane + 64 * (i % PPL), a.cpr - 1);
    buf[i] = pb[static_cast<int64_t>(kk) * a.cpr + cc];
  }
}

// cpr <= 64: the wave's rows are packed 64 / P2 to a register (P2 = cpr
// rounded up to a power of two, lg = log2 P2), so one log2(P2)-step
// reduction merges them all.
__device__ inline void load_packed(const AcceptArgs& a, const AcceptPartial* pb, int nr, int wave,
                                   int lane, int lg, AcceptPartial (&buf)[kFinalRegs]) {
  constexpr int NWV = NT / 64;
  const int R = 64 >> lg;
#pragma unroll
  for (int p = 0; p < kFinalRegs; ++p) {
    const int kk = min(wave + NWV * (p * R + (lane >> lg)), nr - 1);
    const int cc = min(lane & ((1 << lg) - 1), a.cpr - 1);
    buf[p] = pb[static_cast<int64_t>(kk) * a.cpr + cc];
  }
}

__device__ inline void merge_packed(const AcceptArgs& a, int nr, int wave, int lane, int lg, int rpw,
                                    const AcceptPartial (&buf)[kFinalRegs], Best* s_row) {
  constexpr int NWV = NT / 64;
  const int R = 64 >> lg;
#pragma unroll
  for (int p = 0; p < kFinalRegs; ++p) {
    if (p * R >= rpw) break;
    const int kk = wave + NWV * (p * R + (lane >> lg));
    const int cc = lane & ((1 << lg) - 1);
    Best r = {kNegInf, kNoIndex, 0.f};
    if (cc < a.cpr && kk < nr) r = Best{buf[p].mx, buf[p].ix, buf[p].sm};
    for (int sh = (1 << lg) >> 1; sh >= 1; sh >>= 1) {
      Best o;
      o.mx = __shfl_xor(r.mx, sh);
      o.ix = __shfl_xor(r.ix, sh);
      o.sm = __shfl_xor(r.sm, sh);
      r = combine(r, o, a.cl);
    }
    if (cc == 0 && kk < nr) s_row[kk] = r;
  }
}

template <int PPL>
__device__ inline void merge_rows(const AcceptArgs& a, int nr, int wave, int lane,
                                  const AcceptPartial (&buf)[kFinalRegs], Best* s_row) {
  constexpr int NWV = NT / 64;
#pragma unroll
  for (int j = 0; j < kFinalRegs / PPL; ++j) {
    const int kk = wave + NWV * j;
    if (kk >= nr) break;
    Best r = {kNegInf, kNoIndex, 0.f};
#pragma unroll
    for (int q = 0; q < PPL; ++q) {
      const AcceptPartial pr = buf[j * PPL + q];
      if (lane + 64 * q < a.cpr) r = combine(r, Best{pr.mx, pr.ix, pr.sm}, a.cl);
    }
    r = wave_reduce(r, a.cl);
    if (lane == 0) s_row[kk] = r;
  }
}

// One work-group per sequence: merge the chunks of every row, then the
// per-row outputs, draft probabilities and the accepted-prefix length.
// LMHEAD: the logits were never stored; the scan left each drafted token's
// logit in a.xdraft.
template <bool BF16, bool LMHEAD = false>
__global__ void __launch_bounds__(NT) finalize_kernel(AcceptArgs a) {
  constexpr int NWV = NT / 64;
  __shared__ Best s_row[kMaxNew];
  __shared__ int s_step[kMaxNew];
  __shared__ int s_row_of_step[kMaxNew];
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t* step_row = a.step_map + static_cast<int64_t>(b) * a.B;
  const AcceptPartial* pb = a.part + static_cast<int64_t>(b) * a.rows * a.cpr;
  const int esz = BF16 ? 2 : 4;
  const char* logits_b = static_cast<const char*>(a.logits) + static_cast<int64_t>(b) * a.B * a.V * esz;

  // First round of loads, none waiting on another: step map, this lane's
  // draft, and the chunk partials of every row (rows that were not scanned
  // hold stale partials, which are never used).
  // A zero the compiler cannot see through keeps this a vector load issued
  // with the others (as a scalar load it is scheduled after the first wait).
  int lane_zero;
  asm volatile("v_mov_b32 %0, 0" : "=v"(lane_zero));
  const int nref = a.num_ref[b + lane_zero];
  const int step_t = step_row[min(tid, a.B - 1)];
  int tok = -1;
  if (a.L > 0) tok = a.draft_ids[static_cast<int64_t>(b) * a.L + min(lane, a.L - 1)];
  const int rpw = (a.B + NWV - 1) / NWV;     // rows of this wave: wave, wave + NWV, ...
  const int ppl = (a.cpr + 63) / 64;         // partials per lane per row
  const int mode = ppl == 1 && rpw <= kFinalRegs ? 1 : ppl == 2 && 2 * rpw <= kFinalRegs ? 2
                 : ppl <= 4 && 4 * rpw <= kFinalRegs ? 4 : 0;
  const int lg = 32 - __clz(max(a.cpr, 1) - 1);   // ceil(log2(cpr)), <= 6 in mode 1
  AcceptPartial buf[kFinalRegs];
  if (mode == 1) load_packed(a, pb, a.B, wave, lane, lg, buf);
  else if (mode == 2) load_rows<2>(a, pb, a.B, wave, lane, buf);
  else if (mode == 4) load_rows<4>(a, pb, a.B, wave, lane, buf);
  if (tid < a.B) s_step[tid] = step_t;
  if (tid < kMaxNew) s_row_of_step[tid] = -1;
  const int gamma = min(max(nref, 0), a.L);
  __syncthreads();
  if (tid < a.B && step_t >= 1 && step_t <= gamma) s_row_of_step[step_t - 1] = tid;
  __syncthreads();

  // Second round: the drafted token's logit at its verification row.
  const int r = lane;
  int kr = -1;
  float x = 0.f;
  if (wave == 0 && r < gamma) {
    kr = s_row_of_step[r];
    if (kr >= 0 && tok >= 0 && tok < a.V) {
      if (LMHEAD) x = a.xdraft[static_cast<int64_t>(b) * a.L + r];
      else x = load_elem<BF16>(logits_b + static_cast<int64_t>(kr) * a.V * esz, tok);
    }
  }

  if (mode == 1) merge_packed(a, a.B, wave, lane, lg, rpw, buf, s_row);
  else if (mode == 2) merge_rows<2>(a, a.B, wave, lane, buf, s_row);
  else if (mode == 4) merge_rows<4>(a, a.B, wave, lane, buf, s_row);
  else {
    // Many partials per row (the LM-head scan leaves one per vocabulary
    // tile): eight independent loads per lane in flight, then their merge.
    constexpr int U = 8;
    for (int kk = wave; kk < a.B; kk += NWV) {
      Best rr = {kNegInf, kNoIndex, 0.f};
      const AcceptPartial* prow = pb + static_cast<int64_t>(kk) * a.cpr;
      for (int c0 = 0; c0 < a.cpr; c0 += 64 * U) {
        AcceptPartial v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int cc = c0 + 64 * u + lane;
          if (cc < a.cpr) v[u] = prow[cc];
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
          if (c0 + 64 * u + lane < a.cpr) rr = combine(rr, Best{v[u].mx, v[u].ix, v[u].sm}, a.cl);
      }
      rr = wave_reduce(rr, a.cl);
      if (lane == 0) s_row[kk] = rr;
    }
  }
  __syncthreads();
  if (tid < a.B) {
    const bool scanned = s_step[tid] >= 1;
    a.target_ids[static_cast<int64_t>(b) * a.B + tid] = scanned ? s_row[tid].ix : -1;
    if (a.confidence)
      a.confidence[static_cast<int64_t>(b) * a.B + tid] = scanned ? 1.f / s_row[tid].sm : 0.f;
  }
  // One lane per draft r: match flag and probability; the accepted prefix
  // ends at the first rejected draft (a wave ballot).
  if (wave == 0) {
    bool rejected = false;
    float p = 0.f;
    if (r < gamma) {
      rejected = kr < 0 || s_row[kr].ix != tok;
      if (kr >= 0 && tok >= 0 && tok < a.V)
        p = __builtin_amdgcn_exp2f((x - s_row[kr].mx) * a.cl) / s_row[kr].sm;
    }
    if (a.draft_prob && r < a.L) a.draft_prob[static_cast<int64_t>(b) * a.L + r] = p;
    const unsigned long long rej = __ballot(rejected);
    if (lane == 0) a.accept_len[b] = rej ? __ffsll(static_cast<long long>(rej)) - 1 : gamma;
  }
}

// ---- Stochastic acceptance: eq. 2 at temperature T ---------------------------
//
// Draft r is accepted iff u_r * p_phi(D_r) < p_theta(D_r) (probability
// min(1, p_theta / p_phi) for u_r ~ U[0, 1)), in draft order; the accepted
// prefix ends at the first rejection, where the token is drawn from the
// residual max(0, p_theta - p_phi) (or p_theta when that is empty everywhere)
// by inverse CDF in vocabulary order with the uniform w = uniforms[b, L].
// After the scan, accept_sampled_kernel runs draw_chunks work-groups per
// sequence: each merges the chunk partials of the rows it needs and takes the
// acceptance decision (cheap, so every group repeats it), group 0 writes the
// per-draft outputs, and every group sums the residual and p_theta over its
// vocabulary chunk.  draw_pick_kernel (one group per sequence) then finds the
// chunk where the running sum passes w * Z and the entry inside it.

// Weights of the VEC entries of vector v of the draw rows: the residual in q,
// p_theta in t.  Both probabilities are rounded before the difference
// (contraction off: no fused multiply-subtract), so equal distributions leave
// an exactly empty residual and every pass adds the same rounded weights.
template <int VEC>
__device__ inline void draw_weights(const float (&xt)[VEC], const float (&xd)[VEC], const DrawRow& r,
                                    float cl, float (&q)[VEC], float (&t)[VEC]) {
#pragma clang fp contract(off)
#pragma unroll
  for (int e = 0; e < VEC; ++e) {
    t[e] = __builtin_amdgcn_exp2f((xt[e] - r.mt) * cl) * r.ct;
    q[e] = fmaxf(t[e] - __builtin_amdgcn_exp2f((xd[e] - r.md) * cl) * r.cd, 0.f);
  }
}

template <bool BF16>
__device__ inline void draw_rows(const AcceptArgs& a, int b, const DrawRow& r, const char*& trow,
                                 const char*& drow) {
  const int esz = BF16 ? 2 : 4;
  trow = static_cast<const char*>(a.logits) + (static_cast<int64_t>(b) * a.B + r.kr) * a.V * esz;
  drow = static_cast<const char*>(a.draft_logits) + (static_cast<int64_t>(b) * a.L + r.acc) * a.V * esz;
}

template <bool BF16, int VEC>
__global__ void __launch_bounds__(NT) accept_sampled_kernel(AcceptArgs a) {
  constexpr int NWV = NT / 64;
  __shared__ Best s_row[2 * kMaxNew];        // [0, B): verification rows; B + r: draft row r
  __shared__ int s_step[kMaxNew];
  __shared__ int s_row_of_step[kMaxNew];
  __shared__ int s_acc;
  __shared__ float s_sum[2][NWV];
  __shared__ int s_last[2][NWV];
  const int c = blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int esz = BF16 ? 2 : 4;
  const int32_t* step_row = a.step_map + static_cast<int64_t>(b) * a.B;
  const AcceptPartial* pb = a.part + static_cast<int64_t>(b) * a.rows * a.cpr;

  // First round of loads, none waiting on another (see finalize_kernel).
  int lane_zero;
  asm volatile("v_mov_b32 %0, 0" : "=v"(lane_zero));
  const int nref = a.num_ref[b + lane_zero];
  const int step_t = step_row[min(tid, a.B - 1)];
  int tok = -1;
  if (a.L > 0) tok = a.draft_ids[static_cast<int64_t>(b) * a.L + min(lane, a.L - 1)];
  const float u = a.uniforms[static_cast<int64_t>(b) * (a.L + 1) + min(lane, a.L)];
  // The chunk partials of all B + L rows, loaded with the first round as in
  // finalize_kernel (rows this step did not scan hold stale values, unused).
  const int nr = a.B + a.L;
  const int rpw = (nr + NWV - 1) / NWV;
  const int ppl = (a.cpr + 63) / 64;
  const int mode = ppl == 1 && rpw <= kFinalRegs ? 1 : ppl == 2 && 2 * rpw <= kFinalRegs ? 2
                 : ppl <= 4 && 4 * rpw <= kFinalRegs ? 4 : 0;
  const int lg = 32 - __clz(max(a.cpr, 1) - 1);
  AcceptPartial buf[kFinalRegs];
  if (mode == 1) load_packed(a, pb, nr, wave, lane, lg, buf);
  else if (mode == 2) load_rows<2>(a, pb, nr, wave, lane, buf);
  else if (mode == 4) load_rows<4>(a, pb, nr, wave, lane, buf);
  const int gamma = min(max(nref, 0), a.L);
  if (tid < a.B) s_step[tid] = step_t;
  if (tid < kMaxNew) s_row_of_step[tid] = -1;
  __syncthreads();
  if (tid < a.B && step_t >= 1 && step_t <= gamma) s_row_of_step[step_t - 1] = tid;
  if (mode == 1) merge_packed(a, nr, wave, lane, lg, rpw, buf, s_row);
  else if (mode == 2) merge_rows<2>(a, nr, wave, lane, buf, s_row);
  else if (mode == 4) merge_rows<4>(a, nr, wave, lane, buf, s_row);
  else {
    for (int kk = wave; kk < a.B + gamma; kk += NWV) {
      if (kk < a.B && !(s_step[kk] >= 1 && s_step[kk] <= gamma)) continue;
      Best rr = {kNegInf, kNoIndex, 0.f};
      for (int cc = lane; cc < a.cpr; cc += 64) {
        const AcceptPartial pr = pb[static_cast<int64_t>(kk) * a.cpr + cc];
        rr = combine(rr, Best{pr.mx, pr.ix, pr.sm}, a.cl);
      }
      rr = wave_reduce(rr, a.cl);
      if (lane == 0) s_row[kk] = rr;
    }
  }
  __syncthreads();

  const char* lt = static_cast<const char*>(a.logits) + static_cast<int64_t>(b) * a.B * a.V * esz;
  if (wave == 0) {
    // Lane r: the draft's probabilities under both distributions and its test.
    const int r = lane;
    bool rejected = false;
    float pt = 0.f, pd = 0.f;
    if (r < gamma) {
      const int kr = s_row_of_step[r];
      const bool ok = kr >= 0 && tok >= 0 && tok < a.V;
      if (ok) {
        const char* ld = static_cast<const char*>(a.draft_logits) +
                         (static_cast<int64_t>(b) * a.L + r) * a.V * esz;
        const float xt = load_elem<BF16>(lt + static_cast<int64_t>(kr) * a.V * esz, tok);
        const float xd = load_elem<BF16>(ld, tok);
        pt = __builtin_amdgcn_exp2f((xt - s_row[kr].mx) * a.cl) / s_row[kr].sm;
        pd = __builtin_amdgcn_exp2f((xd - s_row[a.B + r].mx) * a.cl) / s_row[a.B + r].sm;
      }
      rejected = !(ok && u * pd < pt);
    }
    const unsigned long long rej = __ballot(rejected);
    const int acc = rej ? __ffsll(static_cast<long long>(rej)) - 1 : gamma;
    if (c == 0) {
      if (r < a.L) {
        if (a.draft_prob) a.draft_prob[static_cast<int64_t>(b) * a.L + r] = pt;
        if (a.p_draft) a.p_draft[static_cast<int64_t>(b) * a.L + r] = pd;
      }
      if (lane == 0) a.accept_len[b] = acc;
    }
    if (lane == 0) s_acc = acc;
  }
  __syncthreads();
  const int acc = s_acc;
  DrawRow dr;
  dr.acc = acc;
  dr.kr = acc < gamma ? s_row_of_step[acc] : -1;
  if (dr.kr < 0) {                             // every draft accepted: no draw
    if (c == 0 && tid == 0) {
      a.correction[b] = -1;
      a.draw_row[b] = dr;
    }
    return;
  }
  dr.mt = s_row[dr.kr].mx;
  dr.ct = 1.f / s_row[dr.kr].sm;
  dr.md = s_row[a.B + acc].mx;
  dr.cd = 1.f / s_row[a.B + acc].sm;
  if (c == 0 && tid == 0) a.draw_row[b] = dr;

  // This group's vocabulary chunk of the draw row: sums and last positive entries.
  const char *trow, *drow;
  draw_rows<BF16>(a, b, dr, trow, drow);
  const int64_t v0 = static_cast<int64_t>(c) * a.draw_vecs, v1 = min(a.nvec, v0 + a.draw_vecs);
  float sq = 0.f, st = 0.f;
  int lq = -1, lt_ = -1;
  for (int64_t v = v0 + tid; v < v1; v += NT) {
    float xt[VEC], xd[VEC], q[VEC], t[VEC];
    load_vec<BF16, VEC>(trow, v, xt);
    load_vec<BF16, VEC>(drow, v, xd);
    draw_weights<VEC>(xt, xd, dr, a.cl, q, t);
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      sq += q[e];
      st += t[e];
      if (q[e] > 0.f) lq = static_cast<int>(v * VEC + e);
      if (t[e] > 0.f) lt_ = static_cast<int>(v * VEC + e);
    }
  }
#pragma unroll
  for (int sh = 32; sh >= 1; sh >>= 1) {
    sq += __shfl_xor(sq, sh);
    st += __shfl_xor(st, sh);
    lq = max(lq, __shfl_xor(lq, sh));
    lt_ = max(lt_, __shfl_xor(lt_, sh));
  }
  if (lane == 0) {
    s_sum[0][wave] = sq;
    s_sum[1][wave] = st;
    s_last[0][wave] = lq;
    s_last[1][wave] = lt_;
  }
  __syncthreads();
  if (tid == 0) {
    DrawPartial dp = {0.f, 0.f, -1, -1};
    for (int i = 0; i < NWV; ++i) {
      dp.sq += s_sum[0][i];
      dp.st += s_sum[1][i];
      dp.lq = max(dp.lq, s_last[0][i]);
      dp.lt = max(dp.lt, s_last[1][i]);
    }
    a.draw_part[static_cast<int64_t>(b) * a.draw_chunks + c] = dp;
  }
}

// Inclusive prefix sums of two values over the work-group's threads (thread
// order).
__device__ inline float2 block_inclusive_scan2(float2 x, float2* s_wave, int lane, int wave) {
  constexpr int NWV = NT / 64;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const float y0 = __shfl_up(x.x, d), y1 = __shfl_up(x.y, d);
    if (lane >= d) {
      x.x += y0;
      x.y += y1;
    }
  }
  if (lane == 63) s_wave[wave] = x;
  __syncthreads();
  float2 base = {0.f, 0.f};
#pragma unroll
  for (int i = 0; i < NWV; ++i)
    if (i < wave) {
      base.x += s_wave[i].x;
      base.y += s_wave[i].y;
    }
  __syncthreads();
  return float2{base.x + x.x, base.y + x.y};
}

// One work-group per sequence with a draw: the chunk where the running sum
// passes w * Z (one prefix sum over the chunk sums), then inside that chunk
// each thread takes a contiguous run of vectors, so one more prefix sum over
// the threads' run sums finds the thread, which walks its run.
template <bool BF16, int VEC>
__global__ void __launch_bounds__(NT) draw_pick_kernel(AcceptArgs a) {
  constexpr int RB = 4;                        // vectors of a run loaded at once
  __shared__ float2 s_wave[NT / 64];
  __shared__ float2 s_tot;
  __shared__ int s_hit, s_last;
  __shared__ float s_base;
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // The chunk partials (draw_chunks <= NT) load with the draw row.
  const DrawPartial* pp = a.draw_part + static_cast<int64_t>(b) * a.draw_chunks;
  DrawPartial mine = {0.f, 0.f, -1, -1};
  if (tid < a.draw_chunks) mine = pp[tid];
  const DrawRow dr = a.draw_row[b];
  const float w = a.uniforms[static_cast<int64_t>(b) * (a.L + 1) + a.L];
  if (dr.kr < 0) return;                       // no draw (correction already -1)

  const float2 incl = block_inclusive_scan2(float2{mine.sq, mine.st}, s_wave, lane, wave);
  if (tid == NT - 1) s_tot = incl;
  if (tid == 0) {
    s_hit = NT;
    s_last = -1;
  }
  __syncthreads();
  const int sel = s_tot.x > 0.f ? 0 : 1;       // empty residual: draw from p_theta
  const float target = w * (sel ? s_tot.y : s_tot.x);
  const float mi = sel ? incl.y : incl.x, my = sel ? mine.st : mine.sq;
  const int mylast = sel ? mine.lt : mine.lq;
  if (tid < a.draw_chunks) {
    if (mi > target) atomicMin(&s_hit, tid);
    atomicMax(&s_last, mylast);
  }
  __syncthreads();
  const int C = s_hit;
  if (C >= a.draw_chunks) {                    // the target rounded onto the total
    if (tid == 0) a.correction[b] = s_last;
    return;
  }
  __syncthreads();
  if (tid == C) {
    s_base = mi - my;
    s_last = mylast;
  }
  __syncthreads();
  const float base = s_base;
  const int clast = s_last;

  // Chunk C: thread tid owns vectors [c0, c1), a contiguous run.
  const char *trow, *drow;
  draw_rows<BF16>(a, b, dr, trow, drow);
  const int64_t v0 = static_cast<int64_t>(C) * a.draw_vecs, v1 = min(a.nvec, v0 + a.draw_vecs);
  const int64_t k = (v1 - v0 + NT - 1) / NT;
  const int64_t c0 = min(v1, v0 + tid * k), c1 = min(v1, c0 + k);
  float ls = 0.f;
  for (int64_t vb = c0; vb < c1; vb += RB) {
    float xt[RB][VEC], xd[RB][VEC];
#pragma unroll
    for (int r = 0; r < RB; ++r)
      if (vb + r < c1) {
        load_vec<BF16, VEC>(trow, vb + r, xt[r]);
        load_vec<BF16, VEC>(drow, vb + r, xd[r]);
      }
#pragma unroll
    for (int r = 0; r < RB; ++r)
      if (vb + r < c1) {
        float q[VEC], t[VEC];
        draw_weights<VEC>(xt[r], xd[r], dr, a.cl, q, t);
#pragma unroll
        for (int e = 0; e < VEC; ++e) ls += sel ? t[e] : q[e];
      }
  }
  const float2 in2 = block_inclusive_scan2(float2{ls, 0.f}, s_wave, lane, wave);
  const float in = base + in2.x;
  if (tid == 0) s_hit = NT;
  __syncthreads();
  if (c0 < c1 && in > target) atomicMin(&s_hit, tid);
  __syncthreads();
  const int T0 = s_hit;
  if (T0 >= NT) {                              // the target rounded past this chunk
    if (tid == 0) a.correction[b] = clast;
    return;
  }
  if (tid != T0) return;
  // Walk the run (its vectors are re-read: cache hits) in the same order.
  float rr = in - ls;
  int x = -1, xl = static_cast<int>(c0 * VEC);
  for (int64_t v = c0; v < c1 && x < 0; ++v) {
    float xt[VEC], xd[VEC], q[VEC], t[VEC];
    load_vec<BF16, VEC>(trow, v, xt);
    load_vec<BF16, VEC>(drow, v, xd);
    draw_weights<VEC>(xt, xd, dr, a.cl, q, t);
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const float wgt = sel ? t[e] : q[e];
      if (wgt > 0.f) xl = static_cast<int>(v * VEC + e);
      rr += wgt;
      if (x < 0 && rr > target) x = static_cast<int>(v * VEC + e);
    }
  }
  a.correction[b] = x >= 0 ? x : xl;
}

}  // namespace

hipError_t launch_accept(const simsd_accept_desc& d, const AcceptPlan& p, const AcceptArgs& a,
                         hipStream_t st) {
  const dim3 grid(p.cpr, d.block_size, d.batch);
  const dim3 block(NT);
  const bool bf16 = d.logits_dtype == SIMSD_BF16;
  if (bf16) {
    if (p.vec == 8) hipLaunchKernelGGL((scan_kernel<true, 8, false>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((scan_kernel<true, 1, false>), grid, block, 0, st, a);
  } else {
    if (p.vec == 4) hipLaunchKernelGGL((scan_kernel<false, 4, false>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((scan_kernel<false, 1, false>), grid, block, 0, st, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (bf16) hipLaunchKernelGGL((finalize_kernel<true>), dim3(d.batch), block, 0, st, a);
  else hipLaunchKernelGGL((finalize_kernel<false>), dim3(d.batch), block, 0, st, a);
  return hipGetLastError();
}

hipError_t launch_finalize_lmhead(int batch, const AcceptArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((finalize_kernel<true, true>), dim3(batch), dim3(NT), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_accept_sampled(const simsd_accept_desc& d, const AcceptPlan& p,
                                 const AcceptArgs& a, hipStream_t st) {
  const dim3 grid(p.cpr, d.block_size + d.max_ref, d.batch);
  const dim3 block(NT);
  const bool bf16 = d.logits_dtype == SIMSD_BF16;
  if (bf16) {
    if (p.vec == 8) hipLaunchKernelGGL((scan_kernel<true, 8, true>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((scan_kernel<true, 1, true>), grid, block, 0, st, a);
  } else {
    if (p.vec == 4) hipLaunchKernelGGL((scan_kernel<false, 4, true>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((scan_kernel<false, 1, true>), grid, block, 0, st, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const dim3 dgrid(p.draw_chunks, d.batch);
  if (bf16) {
    if (p.vec == 8) {
      hipLaunchKernelGGL((accept_sampled_kernel<true, 8>), dgrid, block, 0, st, a);
      hipLaunchKernelGGL((draw_pick_kernel<true, 8>), dim3(d.batch), block, 0, st, a);
    } else {
      hipLaunchKernelGGL((accept_sampled_kernel<true, 1>), dgrid, block, 0, st, a);
      hipLaunchKernelGGL((draw_pick_kernel<true, 1>), dim3(d.batch), block, 0, st, a);
    }
  } else {
    if (p.vec == 4) {
      hipLaunchKernelGGL((accept_sampled_kernel<false, 4>), dgrid, block, 0, st, a);
      hipLaunchKernelGGL((draw_pick_kernel<false, 4>), dim3(d.batch), block, 0, st, a);
    } else {
      hipLaunchKernelGGL((accept_sampled_kernel<false, 1>), dgrid, block, 0, st, a);
      hipLaunchKernelGGL((draw_pick_kernel<false, 1>), dim3(d.batch), block, 0, st, a);
    }
  }
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Allocation-free greedy accept.  The device address of `scratch` is looked up
// once per device (with that device current) and kept; calls then pass it to
// the same kernels simsd_verify_accept launches, in place of the workspace.
// ----------------------------------------------------------------------------
namespace {

constexpr int kScratchDevices = 64;
std::atomic<void*> g_scratch_ptr[kScratchDevices];
std::mutex g_scratch_mu;

hipError_t scratch_address(int dev, void** out) {
  if (dev < 0 || dev >= kScratchDevices) return hipErrorInvalidDevice;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      int cur = 0;
      hipError_t e = hipGetDevice(&cur);
      if (e != hipSuccess) return e;
      if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return e;
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (cur != dev) {
        const hipError_t e2 = hipSetDevice(cur);
        if (e == hipSuccess) e = e2;
      }
      if (e != hipSuccess) return e;
      if (!p) return hipErrorInvalidSymbol;
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return hipSuccess;
}

}  // namespace
}  // namespace simsd

extern "C" simsd_status simsd_verify_accept_noalloc(const simsd_accept_desc* desc,
                                                    const void* logits, const int32_t* draft_ids,
                                                    const int32_t* step_map,
                                                    const int32_t* num_ref, int32_t* target_ids,
                                                    float* confidence, float* draft_prob,
                                                    int32_t* accept_len, void* stream) {
  using namespace simsd;
  try {
    int dev = 0, cus = 0;
    const hipError_t qe = stream_device(stream, &dev, &cus);
    AcceptPlan p;
    simsd_status st = plan_accept(desc, cus, &p);
    if (st != SIMSD_OK) return st;
    if (p.workspace > SIMSD_NOALLOC_SCRATCH_BYTES) {
      set_error("accept_noalloc: this shape needs " + std::to_string(p.workspace) +
                " bytes of scratch, more than the fixed " +
                std::to_string(SIMSD_NOALLOC_SCRATCH_BYTES) +
                "; call simsd_verify_accept with a workspace instead");
      return SIMSD_ERR_WORKSPACE;
    }
    st = check_accept_inputs(desc, logits, draft_ids, step_map, num_ref, target_ids, accept_len);
    if (st != SIMSD_OK) return st;
    void* part = nullptr;
    hipError_t e = qe;
    if (e == hipSuccess) e = scratch_address(dev, &part);
    if (e != hipSuccess) {
      set_error(std::string("simsd_verify_accept_noalloc: device scratch: ") + hipGetErrorString(e));
      return SIMSD_ERR_HIP;
    }
    AcceptArgs a{};
    a.logits = logits;
    a.draft_ids = draft_ids;
    a.step_map = step_map;
    a.num_ref = num_ref;
    a.target_ids = target_ids;
    a.confidence = confidence;
    a.draft_prob = draft_prob;
    a.accept_len = accept_len;
    a.part = static_cast<AcceptPartial*>(part);
    a.nvec = p.nvec;
    a.chunk_vecs = p.chunk_vecs;
    a.B = desc->block_size;
    a.L = desc->max_ref;
    a.V = desc->vocab;
    a.cpr = p.cpr;
    a.rows = p.rows;
    a.cl = kLog2e;
    e = launch_accept(*desc, p, a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) {
      set_error(std::string("simsd_verify_accept_noalloc launch: ") + hipGetErrorString(e));
      return SIMSD_ERR_HIP;
    }
    return SIMSD_OK;
  } catch (...) {
    set_error("simsd_verify_accept_noalloc: internal error");
    return SIMSD_ERR_HIP;
  }
}
