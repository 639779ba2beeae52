// Vocabulary scan and greedy acceptance of SimSD on gfx950.
//
// Eq. 2 at temperature 0 (Sec. 3.2): draft r is accepted while the target's
// argmax at its verification slot equals it, and the longest such prefix is
// kept.  Each logits row of a scanned block slot (step_map >= 1) is split into
// chunks; one work-group streams a chunk with 16-byte loads and keeps, per
// lane, the running maximum, the first vector reaching it and the sum of
// exp(x - max).  Partials are merged in (value desc, index asc) order, so ties
// resolve to the lowest vocabulary index exactly.  A second kernel, one
// work-group per sequence, merges the chunks of all its rows, computes
// confidence and draft probabilities and walks the drafts in step order.
#include "simsd_kernels.h"

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

__device__ inline Best combine(Best a, Best b) {
  const float M = fmaxf(a.mx, b.mx);
  Best r;
  r.mx = M;
  r.ix = a.mx > b.mx ? a.ix : (b.mx > a.mx ? b.ix : min(a.ix, b.ix));
  const float sa = a.mx == kNegInf ? 0.f : a.sm * __builtin_amdgcn_exp2f((a.mx - M) * kLog2e);
  const float sb = b.mx == kNegInf ? 0.f : b.sm * __builtin_amdgcn_exp2f((b.mx - M) * kLog2e);
  r.sm = sa + sb;
  return r;
}

__device__ inline Best wave_reduce(Best v) {
#pragma unroll
  for (int sh = 32; sh >= 1; sh >>= 1) {
    Best o;
    o.mx = __shfl_xor(v.mx, sh);
    o.ix = __shfl_xor(v.ix, sh);
    o.sm = __shfl_xor(v.sm, sh);
    v = combine(v, o);
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
__device__ Best scan_chunk(const void* row, int64_t v0, int64_t v1, int tid, Best* s_red) {
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
        sm = mx == kNegInf ? 0.f : sm * __builtin_amdgcn_exp2f((mx - vm) * kLog2e);
        mx = vm;
        vbest = v + u * NT;
      }
      const float off = mx * kLog2e;
#pragma unroll
      for (int i = 0; i < VEC; ++i) sm += __builtin_amdgcn_exp2f(fmaf(x[u][i], kLog2e, -off));
    }
  }
  for (; v < v1; v += NT) {
    float x[VEC];
    load_vec<BF16, VEC>(row, v, x);
    float vm = x[0];
#pragma unroll
    for (int i = 1; i < VEC; ++i) vm = fmaxf(vm, x[i]);
    if (vm > mx) {
      sm = mx == kNegInf ? 0.f : sm * __builtin_amdgcn_exp2f((mx - vm) * kLog2e);
      mx = vm;
      vbest = v;
    }
    const float off = mx * kLog2e;
#pragma unroll
    for (int i = 0; i < VEC; ++i) sm += __builtin_amdgcn_exp2f(fmaf(x[i], kLog2e, -off));
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
  me = wave_reduce(me);
  const int lane = tid & 63, wave = tid >> 6;
  if (lane == 0) s_red[wave] = me;
  __syncthreads();
  Best r = s_red[0];
  for (int i = 1; i < NT / 64; ++i) r = combine(r, s_red[i]);
  return r;
}

// One work-group per (vocabulary chunk, block slot, sequence): writes the
// chunk's (max, lowest index, sum of exp) to the workspace.
template <bool BF16, int VEC>
__global__ void __launch_bounds__(NT) scan_kernel(AcceptArgs a) {
  __shared__ Best s_red[NT / 64];
  const int c = blockIdx.x, k = blockIdx.y, b = blockIdx.z;
  const int64_t rowi = static_cast<int64_t>(b) * a.B + k;
  if (a.step_map[rowi] < 1) return;          // committed or padding: not scanned
  const int esz = BF16 ? 2 : 4;
  const char* row = static_cast<const char*>(a.logits) + rowi * a.V * esz;
  const int64_t v0 = static_cast<int64_t>(c) * a.chunk_vecs;
  const int64_t v1 = min(a.nvec, v0 + a.chunk_vecs);
  const Best r = scan_chunk<BF16, VEC>(row, v0, v1, threadIdx.x, s_red);
  if (threadIdx.x == 0) {
    AcceptPartial pr;
    pr.mx = r.mx;
    pr.ix = r.ix;
    pr.sm = r.sm;
    pr.pad = 0;
    a.part[rowi * a.cpr + c] = pr;
  }
}

// One work-group per sequence: merge the chunks of every row, then the
// per-row outputs, draft probabilities and the accepted-prefix length.
template <bool BF16>
__global__ void __launch_bounds__(NT) finalize_kernel(AcceptArgs a) {
  __shared__ Best s_row[kMaxNew];
  __shared__ int s_row_of_step[kMaxNew];
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t* step_row = a.step_map + static_cast<int64_t>(b) * a.B;
  const int esz = BF16 ? 2 : 4;
  const char* logits_b = static_cast<const char*>(a.logits) + static_cast<int64_t>(b) * a.B * a.V * esz;
  const AcceptPartial* pb = a.part + static_cast<int64_t>(b) * a.B * a.cpr;
  for (int kk = wave; kk < a.B; kk += NT / 64) {
    Best r = {kNegInf, kNoIndex, 0.f};
    if (step_row[kk] >= 1) {
      for (int cc = lane; cc < a.cpr; cc += 64) {
        const AcceptPartial pr = pb[static_cast<int64_t>(kk) * a.cpr + cc];
        r = combine(r, Best{pr.mx, pr.ix, pr.sm});
      }
      r = wave_reduce(r);
    }
    if (lane == 0) s_row[kk] = r;
  }
  const int gamma = min(max(a.num_ref[b], 0), a.L);
  if (tid < kMaxNew) s_row_of_step[tid] = -1;
  __syncthreads();
  if (tid < a.B) {
    const int s = step_row[tid];
    if (s >= 1 && s <= gamma) s_row_of_step[s - 1] = tid;
    const bool scanned = s >= 1;
    a.target_ids[static_cast<int64_t>(b) * a.B + tid] = scanned ? s_row[tid].ix : -1;
    if (a.confidence)
      a.confidence[static_cast<int64_t>(b) * a.B + tid] = scanned ? 1.f / s_row[tid].sm : 0.f;
  }
  __syncthreads();
  // One lane per draft r: its verification row, match flag and probability.
  // The accepted prefix ends at the first rejected draft (a wave ballot).
  if (wave == 0) {
    const int r = lane;
    bool rejected = false;
    float p = 0.f;
    if (r < gamma) {
      const int kr = s_row_of_step[r];
      const int tok = a.draft_ids[static_cast<int64_t>(b) * a.L + r];
      rejected = kr < 0 || s_row[kr].ix != tok;
      if (kr >= 0 && tok >= 0 && tok < a.V) {
        const float x = load_elem<BF16>(logits_b + static_cast<int64_t>(kr) * a.V * esz, tok);
        p = __builtin_amdgcn_exp2f((x - s_row[kr].mx) * kLog2e) / s_row[kr].sm;
      }
    }
    if (a.draft_prob && r < a.L) a.draft_prob[static_cast<int64_t>(b) * a.L + r] = p;
    const unsigned long long rej = __ballot(rejected);
    if (lane == 0) a.accept_len[b] = rej ? __ffsll(static_cast<long long>(rej)) - 1 : gamma;
  }
}

}  // namespace

hipError_t launch_accept(const simsd_accept_desc& d, const AcceptPlan& p, const AcceptArgs& a,
                         hipStream_t st) {
  const dim3 grid(p.cpr, d.block_size, d.batch);
  const dim3 block(NT);
  const bool bf16 = d.logits_dtype == SIMSD_BF16;
  if (bf16) {
    if (p.vec == 8) hipLaunchKernelGGL((scan_kernel<true, 8>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((scan_kernel<true, 1>), grid, block, 0, st, a);
  } else {
    if (p.vec == 4) hipLaunchKernelGGL((scan_kernel<false, 4>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((scan_kernel<false, 1>), grid, block, 0, st, a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (bf16) hipLaunchKernelGGL((finalize_kernel<true>), dim3(d.batch), block, 0, st, a);
  else hipLaunchKernelGGL((finalize_kernel<false>), dim3(d.batch), block, 0, st, a);
  return hipGetLastError();
}

}  // namespace simsd
