// LM-head product fused with the vocabulary scan of SimSD's greedy acceptance
// on gfx950.
//
// Sec. 3.2: the target distribution at a verification slot is the target
// model's prediction there, the LM head applied to the slot's final hidden
// state.  lmhead_scan_kernel computes those logits tile by tile on the matrix
// cores -- logits^T[vocab, row] = W[vocab, :] . hidden[row, :]^T with
// v_mfma_f32_32x32x16_bf16 -- and reduces each row over each 128- or 256-entry
// vocabulary tile to (max, lowest index reaching it, sum of exp(x - max)) in
// the epilogue, the partial the logits scan writes, so the logits never reach
// memory.  The tile that holds a row's drafted token also stores that logit
// for the draft probability.  lmhead_merge_kernel merges each row's partials
// (one wave per row) and finalize_kernel (simsd_accept.hip) finds the accepted
// prefix from them as for stored logits.
//
// Tiles: TR rows x TV vocabulary entries per work-group of WV x WR waves (4 x 2
// in every variant); wave w covers rows (TR/WR)*(w/WV).. and vocabulary
// (TV/WV)*(w%WV).. in 32 x 32 MFMA blocks.  The reduction dimension streams in
// KS-wide stages through a ring of NBUF LDS stages filled by direct
// global-to-LDS loads, so several stages are in flight without staging
// registers.  A stage row holds CPR 16-byte chunks; chunk c of row r sits at
// position c ^ swz(r), so the operand reads of 16 consecutive rows touch 64
// distinct banks.  Each wave reads the operands of the next 16-wide sub-step
// (across the stage barrier too) while the MFMAs of the current one run.
#include "simsd_kernels.h"

namespace simsd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr int kNoIndex = 0x7fffffff;
constexpr int NT = 512;                  // threads of the merge kernel
// Row-count thresholds of the variants (see launch_lmhead_scan).
constexpr int kFewRows = 32;
constexpr int kOneTileRows = 128;

#define LM_LDS __attribute__((address_space(3)))

// 16 bytes per lane from a per-lane address into LDS at m0 + 16 * lane.
__device__ inline void dma16(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds)) : "memory");
}
// The same with the non-temporal hint: the line is streamed through the L2
// rather than kept there.
__device__ inline void dma16_nt(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off nt"
               :: "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds)) : "memory");
}
template <int N>
__device__ inline void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

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

// TR rows and TV vocabulary entries per tile, KS reduction elements per
// stage, NBUF stages in the ring; WV x WR waves (vocabulary parts x row parts).
// STREAMW: the weight is loaded with the non-temporal hint.
template <int TR, int TV, int KS, int NBUF, int WV, int WR, bool STREAMW>
__global__ void __launch_bounds__(64 * WV * WR) lmhead_scan_kernel(LmheadArgs a) {
  constexpr int NT = 64 * WV * WR;
  constexpr int RBW = TR / (32 * WR);      // 32-row MFMA blocks per wave
  constexpr int VBW = TV / (32 * WV);      // 32-entry MFMA blocks per wave
  constexpr int CPR = KS / 8;              // 16-byte chunks per row per stage
  constexpr int ROWB = KS * 2;             // LDS bytes per row per stage
  constexpr int RPS = 16 / CPR;            // rows spanning the 64 banks
  constexpr int STAGEB = (TV + TR) * ROWB; // one stage: weight rows, then hidden rows
  constexpr int INSN = STAGEB / 1024;      // 1 KB direct loads per stage
  constexpr int PERW = INSN / (NT / 64);   // per wave
  constexpr int RPI = 64 / CPR;            // rows per direct load
  static_assert(RBW >= 1 && TR % (32 * WR) == 0 && VBW >= 1 && TV % (32 * WV) == 0, "wave grid");
  static_assert(KS % 16 == 0 && CPR <= 16, "stage width");
  static_assert(INSN % (NT / 64) == 0, "stage loads split evenly over the waves");
  static_assert(NBUF >= 2 && NBUF <= 5, "ring depth");
  auto swz = [](int r) { return (r / RPS) % CPR; };
  __shared__ __attribute__((aligned(1024))) uint8_t s_ring[NBUF][STAGEB];
  __shared__ Best s_part[WV][TR];         // per vocabulary part, per row of the tile
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n = lane & 31, h = lane >> 5;
  const int rw = wave / WV, vq = wave % WV;
  // Work-groups go to the eight XCDs round-robin.  Tile t = xcd * per + j
  // (row tiles fastest) keeps the row tiles of one vocabulary tile on one XCD,
  // whose L2 then serves them the weight tile once; ids past the last tile
  // (grid padded to a multiple of 8) leave at once.
  const int rtiles = (a.R + TR - 1) / TR, ntiles = rtiles * a.vtiles;
  const int per = (ntiles + 7) / 8;
  const int t = static_cast<int>(blockIdx.x % 8) * per + static_cast<int>(blockIdx.x / 8);
  if (t >= ntiles) return;
  const int vt = t / rtiles;
  const int r0 = (t % rtiles) * TR, v0 = vt * TV;
  const int64_t rowb = static_cast<int64_t>(a.H) * 2;   // bytes per hidden / weight row

  // Instruction g = wave * PERW + i of a stage moves stage rows RPI*g ..
  // RPI*g + RPI-1 (weight rows first, then hidden rows); lane l takes row
  // RPI*g + l/CPR, chunk position l%CPR, i.e. logical chunk (l%CPR) ^ swz(row).
  // Rows past the end read the last row (their results are dropped).
  const char* src[PERW];
  uint32_t dst[PERW];
#pragma unroll
  for (int i = 0; i < PERW; ++i) {
    const int g = wave * PERW + i, r = RPI * g + lane / CPR;
    const int c = (lane % CPR) ^ swz(r);
    const char* rowp = r < TV
        ? static_cast<const char*>(a.weight) + min(v0 + r, a.V - 1) * rowb
        : static_cast<const char*>(a.hidden) + min(r0 + r - TV, a.R - 1) * rowb;
    src[i] = rowp + 16 * c;
    dst[i] = 1024u * g;
  }
  const uint32_t ring0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(
      (LM_LDS void*)(&s_ring[0][0])));
  auto issue = [&](int s) __attribute__((always_inline)) {
    const int64_t off = static_cast<int64_t>(s) * KS * 2;
    const uint32_t slot = ring0 + (s % NBUF) * STAGEB;
#pragma unroll
    for (int i = 0; i < PERW; ++i) {
      if (STREAMW && RPI * (wave * PERW + i) < TV) dma16_nt(src[i] + off, slot + dst[i]);
      else dma16(src[i] + off, slot + dst[i]);
    }
  };

  f32x16 acc[VBW][RBW];                    // [vocab block][row block]
#pragma unroll
  for (int vb = 0; vb < VBW; ++vb)
#pragma unroll
    for (int rb = 0; rb < RBW; ++rb)
#pragma unroll
      for (int j = 0; j < 16; ++j) acc[vb][rb][j] = 0.f;

  // Operand reads: row n of a 32-row block, logical chunk 2*ks + h.
  constexpr int KSUB = KS / 16;
  int ao[KSUB][VBW], bo[KSUB][RBW];
#pragma unroll
  for (int ks = 0; ks < KSUB; ++ks) {
#pragma unroll
    for (int vb = 0; vb < VBW; ++vb) {
      const int rv = (TV / WV) * vq + 32 * vb + n;
      ao[ks][vb] = rv * ROWB + 16 * ((2 * ks + h) ^ swz(rv));
    }
#pragma unroll
    for (int rb = 0; rb < RBW; ++rb) {
      const int rr = TV + (TR / WR) * rw + 32 * rb + n;
      bo[ks][rb] = rr * ROWB + 16 * ((2 * ks + h) ^ swz(rr));
    }
  }

  const int S = a.H / KS;
#pragma unroll
  for (int s = 0; s < NBUF - 1; ++s)
    if (s < S) issue(s);
  // Stage s is waited for, and the ring slot of stage s - 1 refilled, once
  // every wave has passed the barrier.
  auto enter_stage = [&](int s) __attribute__((always_inline)) {
    // Stages issued: 0 .. min(S, s + NBUF - 1) - 1; stage s has landed once
    // at most the younger ones remain.
    const int younger = min(S, s + NBUF - 1) - 1 - s;
    if (NBUF > 4 && younger >= 3) wait_vm<3 * PERW>();
    else if (NBUF > 3 && younger >= 2) wait_vm<2 * PERW>();
    else if (NBUF > 2 && younger >= 1) wait_vm<PERW>();
    else wait_vm<0>();
    lds_barrier();                         // stage s is in; stage s - 1's slot is free
    if (s + NBUF - 1 < S) issue(s + NBUF - 1);
  };
  auto stage_at = [&](int s) __attribute__((always_inline)) {
    return reinterpret_cast<const LM_LDS uint8_t*>(ring0) + (s % NBUF) * STAGEB;
  };
  // Operand fragments in two register sets: the reads of sub-step ks + 1 (or
  // of the next stage's first sub-step) are in flight while the MFMAs of
  // sub-step ks run.
  static_assert(KSUB % 2 == 0, "sub-steps alternate between two fragment sets");
  bf16x8 fa[2][VBW], fb[2][RBW];
  auto read_frags = [&](const LM_LDS uint8_t* st, int ks, int set) __attribute__((always_inline)) {
#pragma unroll
    for (int vb = 0; vb < VBW; ++vb) fa[set][vb] = *reinterpret_cast<const LM_LDS bf16x8*>(st + ao[ks][vb]);
#pragma unroll
    for (int rb = 0; rb < RBW; ++rb) fb[set][rb] = *reinterpret_cast<const LM_LDS bf16x8*>(st + bo[ks][rb]);
  };
  auto mfmas = [&](int set) __attribute__((always_inline)) {
#pragma unroll
    for (int vb = 0; vb < VBW; ++vb)
#pragma unroll
      for (int rb = 0; rb < RBW; ++rb)
        acc[vb][rb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[set][vb], fb[set][rb], acc[vb][rb], 0, 0, 0);
  };
  if (S > 0) {
    enter_stage(0);
    read_frags(stage_at(0), 0, 0);
  }
  for (int s = 0; s < S; ++s) {
    const LM_LDS uint8_t* st = stage_at(s);
#pragma unroll
    for (int ks = 0; ks < KSUB - 1; ++ks) {
      read_frags(st, ks + 1, (ks + 1) & 1);
      mfmas(ks & 1);
    }
    // The last sub-step's fragments are in registers, so the barrier that
    // enters the next stage may pass before its MFMAs issue.
    if (s + 1 < S) {
      enter_stage(s + 1);
      read_frags(stage_at(s + 1), 0, 0);
    }
    mfmas(1);
  }

  // Epilogue.  Register j of acc[vb][rb] holds vocabulary entry
  // v0 + (TV/WV)*vq + 32*vb + 8*(j/4) + 4*h + j%4 of row r0 + (TR/WR)*rw + 32*rb + n.
#pragma unroll
  for (int rb = 0; rb < RBW; ++rb) {
    const int rowl = (TR / WR) * rw + 32 * rb + n, row = r0 + rowl;
    float xv[VBW][16];
#pragma unroll
    for (int vb = 0; vb < VBW; ++vb)
#pragma unroll
      for (int j = 0; j < 16; ++j) xv[vb][j] = acc[vb][rb][j];
    // The drafted token of this row, if it is a verification row.
    int tok = -1, slot = -1;
    if (row < a.R) {
      const int b = row / a.B;
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
    for (int vb = 0; vb < VBW; ++vb)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int v = v0 + (TV / WV) * vq + 32 * vb + 8 * (j >> 2) + 4 * h + (j & 3);
        const float x = xv[vb][j];
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
      for (int vb = 0; vb < VBW; ++vb)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int v = v0 + (TV / WV) * vq + 32 * vb + 8 * (j >> 2) + 4 * h + (j & 3);
          if (v < a.V) sm += __builtin_amdgcn_exp2f((xv[vb][j] - mx) * kLog2e);
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
    for (int q = 1; q < WV; ++q) r = combine(r, s_part[q][tid]);
    AcceptPartial pr;
    pr.mx = r.mx;
    pr.ix = r.ix;
    pr.sm = r.sm;
    pr.pad = 0;
    a.part[static_cast<int64_t>(r0 + tid) * a.vtiles + vt] = pr;
  }
}

// WPR waves per row merge the row's partials, one per vocabulary tile, so the
// finalize kernel (one work-group per sequence) reads a single partial per row.
// WPR = 8 (a work-group per row) for few rows, else one wave per row.
template <int WPR>
__global__ void __launch_bounds__(NT) lmhead_merge_kernel(LmheadArgs a) {
  constexpr int U = 8;                     // loads per lane in flight
  constexpr int NW = NT / 64;
  __shared__ Best s_w[NW];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row = blockIdx.x * (NW / WPR) + wave / WPR;
  if (WPR == 1 && row >= a.R) return;
  Best r = {kNegInf, kNoIndex, 0.f};
  if (row < a.R) {
    const AcceptPartial* pr = a.part + static_cast<int64_t>(row) * a.vtiles;
    for (int c0 = 64 * (wave % WPR) + lane; c0 < a.vtiles; c0 += 64 * WPR * U) {
      AcceptPartial v[U];
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (c0 + 64 * WPR * u < a.vtiles) v[u] = pr[c0 + 64 * WPR * u];
#pragma unroll
      for (int u = 0; u < U; ++u)
        if (c0 + 64 * WPR * u < a.vtiles) r = combine(r, Best{v[u].mx, v[u].ix, v[u].sm});
    }
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) {
      Best o;
      o.mx = __shfl_xor(r.mx, off);
      o.ix = __shfl_xor(r.ix, off);
      o.sm = __shfl_xor(r.sm, off);
      r = combine(r, o);
    }
  }
  if (WPR > 1) {                           // one row per work-group: combine its waves
    if (lane == 0) s_w[wave] = r;
    __syncthreads();
    if (threadIdx.x != 0 || row >= a.R) return;
    r = s_w[0];
#pragma unroll
    for (int w = 1; w < NW; ++w) r = combine(r, s_w[w]);
  } else if (lane != 0) {
    return;
  }
  AcceptPartial m;
  m.mx = r.mx;
  m.ix = r.ix;
  m.sm = r.sm;
  m.pad = 0;
  a.merged[row] = m;
}

}  // namespace

namespace {
template <int TR, int TV, int KS, int NBUF, int WV = 4, int WR = 2, bool STREAMW = false>
hipError_t launch_variant(const LmheadArgs& a, hipStream_t st) {
  if (a.vtiles != (a.V + TV - 1) / TV) return hipErrorInvalidValue;   // plan and launch disagree
  const int ntiles = (a.R + TR - 1) / TR * a.vtiles;
  hipLaunchKernelGGL((lmhead_scan_kernel<TR, TV, KS, NBUF, WV, WR, STREAMW>), dim3((ntiles + 7) / 8 * 8),
                     dim3(64 * WV * WR), 0, st, a);
  return hipGetLastError();
}
}  // namespace

hipError_t launch_lmhead_scan(const LmheadArgs& a, hipStream_t st) {
  // Few rows: the weight stream is all there is; 128-entry vocabulary tiles
  // (more, shorter work-groups) and 54 KB of LDS, two work-groups per CU.  Up
  // to one row tile: 128-byte row segments, one work-group per CU, and the
  // weight (read by no other work-group) streamed past the L2 so that the
  // L2 keeps the hidden rows every work-group re-reads.  More rows: 256-row
  // tiles halve the weight re-reads and the LDS reads per MFMA; the two row
  // tiles of a vocabulary tile share its weight lines through the L2.
  if (a.R <= kFewRows) return launch_variant<128, 128, 32, 3>(a, st);
  if (a.R <= kOneTileRows) return launch_variant<128, 256, 64, 3, 4, 2, true>(a, st);
  return launch_variant<256, 256, 64, 2>(a, st);
}

hipError_t launch_lmhead_merge(const LmheadArgs& a, hipStream_t st) {
  if (a.R <= kFewRows)
    hipLaunchKernelGGL(lmhead_merge_kernel<NT / 64>, dim3(a.R), dim3(NT), 0, st, a);
  else
    hipLaunchKernelGGL(lmhead_merge_kernel<1>, dim3((a.R + NT / 64 - 1) / (NT / 64)), dim3(NT), 0,
                       st, a);
  return hipGetLastError();
}

int lmhead_vocab_tile(int rows) { return rows <= kFewRows ? 128 : 256; }
int lmhead_stage() { return 64; }   // the widest stage of the variants

}  // namespace simsd
