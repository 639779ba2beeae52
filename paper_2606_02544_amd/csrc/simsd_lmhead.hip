// LM-head product fused with the vocabulary scan of SimSD's greedy acceptance
// on gfx950.
//
// Sec. 3.2: the target distribution at a verification slot is the target
// model's prediction there, the LM head applied to the slot's final hidden
// state.  lmhead_scan_kernel computes those logits tile by tile on the matrix
// cores -- logits^T[vocab, row] = W[vocab, :] . hidden[row, :]^T with
// v_mfma_f32_32x32x16_bf16 -- and reduces each row over each 256-entry
// vocabulary tile to (max, lowest index reaching it, sum of exp(x - max)) in
// the epilogue, the partial the logits scan writes, so the logits never reach
// memory.  The tile that holds a row's drafted token also stores that logit
// for the draft probability.  finalize_kernel (simsd_accept.hip) then merges
// the partials and finds the accepted prefix as for stored logits.
//
// Tiles: 128 rows x 256 vocabulary entries per 8-wave work-group; wave w
// covers rows 64*(w/4).. and vocabulary 64*(w%4).. (2 x 2 MFMA blocks).  The
// reduction dimension streams in 64-wide stages through two LDS buffers
// (register-staged loads of stage s+1 overlap the MFMAs of stage s); rows are
// padded to 144 bytes so the 16-byte operand reads of 32 rows hit distinct
// banks.
#include "simsd_kernels.h"

namespace simsd {
namespace {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kNoIndex = 0x7fffffff;
constexpr int NT = 512;                  // 8 waves
constexpr int TR = 128;                  // rows per tile
constexpr int TV = 256;                  // vocabulary entries per tile
constexpr int KS = 64;                   // reduction elements per stage
constexpr int PITCH = KS * 2 + 16;       // LDS bytes per row (padded)
constexpr int CPR = KS * 2 / 16;         // 16-byte chunks per row per stage
constexpr int WCH = TV * CPR / NT;       // weight chunks per thread per stage
constexpr int HCH = TR * CPR / NT;       // hidden chunks per thread per stage

struct Best {
  float mx;
  int ix;
  float sm;
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

__global__ void __launch_bounds__(NT) lmhead_scan_kernel(LmheadArgs a) {
  __shared__ __attribute__((aligned(16))) uint8_t s_w[2][TV * PITCH];
  __shared__ __attribute__((aligned(16))) uint8_t s_h[2][TR * PITCH];
  __shared__ Best s_part[4][TR];          // per vocabulary quarter, per row of the tile
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31, h = lane >> 5;
  const int rw = wave / 4, vq = wave % 4;
  const int r0 = blockIdx.x * TR, v0 = blockIdx.y * TV;
  const int64_t rowb = static_cast<int64_t>(a.H) * 2;   // bytes per hidden / weight row

  // This thread's chunks of each stage: chunk c = tid + NT*i covers row c/CPR,
  // bytes 16*(c%CPR) of the stage.  Rows past the end read the last row.
  const char* gw[WCH];
  const char* gh[HCH];
  uint32_t lw[WCH], lh[HCH];
#pragma unroll
  for (int i = 0; i < WCH; ++i) {
    const int c = tid + NT * i, r = c / CPR, q = c % CPR;
    gw[i] = static_cast<const char*>(a.weight) + min(v0 + r, a.V - 1) * rowb + 16 * q;
    lw[i] = r * PITCH + 16 * q;
  }
#pragma unroll
  for (int i = 0; i < HCH; ++i) {
    const int c = tid + NT * i, r = c / CPR, q = c % CPR;
    gh[i] = static_cast<const char*>(a.hidden) + min(r0 + r, a.R - 1) * rowb + 16 * q;
    lh[i] = r * PITCH + 16 * q;
  }
  u32x4 rw_[WCH], rh_[HCH];
  auto load_stage = [&](int s) __attribute__((always_inline)) {
    const int64_t off = static_cast<int64_t>(s) * KS * 2;
#pragma unroll
    for (int i = 0; i < WCH; ++i) rw_[i] = *reinterpret_cast<const u32x4*>(gw[i] + off);
#pragma unroll
    for (int i = 0; i < HCH; ++i) rh_[i] = *reinterpret_cast<const u32x4*>(gh[i] + off);
  };
  auto store_stage = [&](int buf) __attribute__((always_inline)) {
#pragma unroll
    for (int i = 0; i < WCH; ++i) *reinterpret_cast<u32x4*>(&s_w[buf][lw[i]]) = rw_[i];
#pragma unroll
    for (int i = 0; i < HCH; ++i) *reinterpret_cast<u32x4*>(&s_h[buf][lh[i]]) = rh_[i];
  };

  f32x16 acc[2][2];                        // [vocab block][row block]
#pragma unroll
  for (int vb = 0; vb < 2; ++vb)
#pragma unroll
    for (int rb = 0; rb < 2; ++rb)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[vb][rb][j] = 0.f;

  const int S = a.H / KS;
  load_stage(0);
  store_stage(0);
  __syncthreads();
  for (int s = 0; s < S; ++s) {
    const int buf = s & 1;
    if (s + 1 < S) load_stage(s + 1);
    const uint8_t* bw = s_w[buf];
    const uint8_t* bh = s_h[buf];
#pragma unroll
    for (int ks = 0; ks < KS / 16; ++ks) {
      const int co = 32 * ks + 16 * h;     // bytes of reduction elements 16*ks + 8*h ..
      bf16x8 fa[2], fb[2];
#pragma unroll
      for (int vb = 0; vb < 2; ++vb)
        fa[vb] = *reinterpret_cast<const bf16x8*>(bw + (64 * vq + 32 * vb + n) * PITCH + co);
#pragma unroll
      for (int rb = 0; rb < 2; ++rb)
        fb[rb] = *reinterpret_cast<const bf16x8*>(bh + (64 * rw + 32 * rb + n) * PITCH + co);
#pragma unroll
      for (int vb = 0; vb < 2; ++vb)
#pragma unroll
        for (int rb = 0; rb < 2; ++rb)
          acc[vb][rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[vb], fb[rb], acc[vb][rb], 0, 0, 0);
    }
    if (s + 1 < S) store_stage(buf ^ 1);
    __syncthreads();
  }

  // Epilogue.  Register j of acc[vb][rb] holds vocabulary entry
  // v0 + 64*vq + 32*vb + 8*(j/4) + 4*h + j%4 of row r0 + 64*rw + 32*rb + n.
#pragma unroll
  for (int rb = 0; rb < 2; ++rb) {
    const int rowl = 64 * rw + 32 * rb + n, row = r0 + rowl;
    // The drafted token of this row, if it is a verification row.
    int tok = -1, slot = -1;
    if (row < a.R) {
      const int b = row / a.B, k = row % a.B;
      const int step = a.step_map[row];
      const int gamma = min(max(a.num_ref[b], 0), a.L);
      if (step >= 1 && step <= gamma) {
        slot = b * a.L + step - 1;
        tok = a.draft_ids[slot];
      }
    }
    float mx = kNegInf;
    int ix = kNoIndex;
#pragma unroll
    for (int vb = 0; vb < 2; ++vb)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int v = v0 + 64 * vq + 32 * vb + 8 * (j >> 2) + 4 * h + (j & 3);
        const float x = acc[vb][rb][j];
        if (v < a.V) {
          if (x > mx || (x == mx && v < ix)) {
            mx = x;
            ix = v;
          }
          if (v == tok) a.xdraft[slot] = x;
        }
      }
    float sm = 0.f;
    if (mx != kNegInf) {
#pragma unroll
      for (int vb = 0; vb < 2; ++vb)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int v = v0 + 64 * vq + 32 * vb + 8 * (j >> 2) + 4 * h + (j & 3);
          if (v < a.V) sm += __builtin_amdgcn_exp2f((acc[vb][rb][j] - mx) * kLog2e);
        }
    }
    Best me = {mx, ix, sm};
    Best other;
    other.mx = __shfl_xor(me.mx, 32);
    other.ix = __shfl_xor(me.ix, 32);
    other.sm = __shfl_xor(me.sm, 32);
    me = combine(me, other);
    if (h == 0) s_part[vq][rowl] = me;
  }
  __syncthreads();
  if (tid < TR && r0 + tid < a.R) {
    Best r = s_part[0][tid];
#pragma unroll
    for (int q = 1; q < 4; ++q) r = combine(r, s_part[q][tid]);
    AcceptPartial pr;
    pr.mx = r.mx;
    pr.ix = r.ix;
    pr.sm = r.sm;
    pr.pad = 0;
    a.part[static_cast<int64_t>(r0 + tid) * a.vtiles + blockIdx.y] = pr;
  }
}

}  // namespace

hipError_t launch_lmhead_scan(const LmheadArgs& a, hipStream_t st) {
  const dim3 grid((a.R + TR - 1) / TR, a.vtiles);
  hipLaunchKernelGGL(lmhead_scan_kernel, grid, dim3(NT), 0, st, a);
  return hipGetLastError();
}

int lmhead_vocab_tile() { return TV; }
int lmhead_stage() { return KS; }

}  // namespace simsd
