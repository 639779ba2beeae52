// Verification attention of SimSD on gfx950 (CDNA4).
//
// Every new slot of a sequence (B block slots, then L reference slots holding
// the drafts) attends to the cached prefix and to the new slots the token-level
// temporal mask allows (Sec. 3.1, eq. 1; verification layout Sec. 3.2).  The
// prefix is visible to every non-padded row; the mask over the new slots is
// built per work-group from the step map as one 64-bit word per row, never
// stored in memory.
//
// Work decomposition: one work-group per (prefix chunk, KV head x row block,
// sequence).  The G query heads of a KV head and all B+L new slots are packed
// into the M rows of one row block (GQA packing), so each K/V byte of the
// prefix is read from HBM once per KV head.  Chunks of one (sequence, KV head,
// row block) write unnormalised partial outputs plus their running max and
// sum; the last chunk to finish (counted with a per-pair ticket) merges them.
//
// bf16 path: K and V tiles of 64 keys are staged through LDS.  Scores are
// computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16, so lane l
// owns query row l % 32 of its wave's 32-row block: the softmax state of a row
// never leaves its two lanes (l, l ^ 32).  The PV product is likewise
// transposed, O^T = V^T P^T, with P taken straight from the score registers as
// the B operand; V is transposed on the fly (8 key rows x DPL dims per lane,
// byte-permuted in registers).  Row maxima are kept in log2 units and only
// rescaled when they grow by more than 2^8 (the exponentials stay <= 256).
#include "simsd_kernels.h"

namespace simsd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLn2 = 0.69314718055994531f;
constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLazy = 8.0f;

// ----------------------------------------------------------------------------
// Temporal mask (Sec. 3.1, eq. 1).  Section 0 = block slot (mask section),
// 1 = reference slot (data section), -1 = padding.  Committed block slots
// (label 0) are visible to every non-padded row; undrafted ones carry label
// gamma + 1.
// ----------------------------------------------------------------------------
struct SlotLabel {
  int sec;
  int tau;
};

__device__ inline SlotLabel slot_label(int slot, const int32_t* step_row, int gamma, int B) {
  if (slot < B) {
    const int s = step_row[slot];
    if (s < 0) return {-1, -1};
    return {0, s > gamma ? gamma + 1 : s};
  }
  const int r = slot - B;
  if (r >= gamma) return {-1, -1};
  return {1, r + 1};
}

// Bit j is set iff new row i may attend to new slot j.  Zero for padding rows.
__device__ uint64_t visibility_word(int i, const int32_t* step_row, int gamma, int B, int n_new) {
  const SlotLabel li = slot_label(i, step_row, gamma, B);
  if (li.sec < 0) return 0ull;
  uint64_t w = 0ull;
  for (int j = 0; j < n_new; ++j) {
    const SlotLabel lj = slot_label(j, step_row, gamma, B);
    bool v;
    if (lj.sec < 0)
      v = false;
    else if (lj.sec == 0 && lj.tau == 0)
      v = true;
    else if (li.sec == 1)
      v = (lj.sec == 1) ? (lj.tau <= li.tau) : (lj.tau > li.tau);
    else
      v = (lj.sec == 1) ? (lj.tau < li.tau) : (lj.tau >= li.tau);
    w |= static_cast<uint64_t>(v) << j;
  }
  return w;
}

__device__ inline uint32_t bf16_bits(float x) {
  return static_cast<uint32_t>(__builtin_bit_cast(uint16_t, static_cast<__bf16>(x)));
}
__device__ inline uint32_t pack_bf16x2(float lo, float hi) {
  return bf16_bits(lo) | (bf16_bits(hi) << 16);
}

// Common prologue: which prefix keys this work-group owns.
struct Work {
  int split, kvh, rb, b, plen, nsplit, kbeg, kend, gamma;
};

__device__ inline bool setup_work(const AttnArgs& a, Work& w) {
  w.split = blockIdx.x;
  w.kvh = blockIdx.y / a.row_blocks;
  w.rb = blockIdx.y % a.row_blocks;
  w.b = blockIdx.z;
  w.plen = min(max(a.prefix_lens[w.b], 0), a.max_prefix);
  w.nsplit = w.plen > 0 ? (w.plen + a.chunk - 1) / a.chunk : 1;
  if (w.split >= w.nsplit) return false;
  w.kbeg = w.split * a.chunk;
  w.kend = min(w.plen, w.kbeg + a.chunk);
  w.gamma = min(max(a.num_ref[w.b], 0), a.L);
  return true;
}

// Element offset of (token key, head kvh, element e) of the cached prefix.
template <bool PAGED>
__device__ inline int64_t cache_offset(const AttnArgs& a, int b, int kvh, int key, int e) {
  int64_t off;
  if (PAGED) {
    const int64_t page = a.block_table[static_cast<int64_t>(b) * a.max_pages + key / a.page_size];
    off = page * a.cs_seq + static_cast<int64_t>(key % a.page_size) * a.cs_tok;
  } else {
    off = static_cast<int64_t>(b) * a.cs_seq + static_cast<int64_t>(key) * a.cs_tok;
  }
  return off + static_cast<int64_t>(kvh) * a.cs_head + e;
}

// Merge of the split partials of one (sequence, KV head, row block), run by
// the last work-group to finish.  Partial layout per split: O[rows_pb][D]
// (unnormalised), then m[rows_pb] (log2 units), then l[rows_pb].
template <int D, int NT, typename OutT>
__device__ void merge_splits(const AttnArgs& a, int64_t pair, const Work& w, const uint64_t* vis,
                             int tid) {
  constexpr int D4 = D / 4;
  const int64_t pstride = static_cast<int64_t>(a.rows_pb) * (D + 2);
  const float* base = a.part + pair * a.splits * pstride;
  const int mo = a.rows_pb * D;
  for (int idx = tid; idx < a.rows_pb * D4; idx += NT) {
    const int rowl = idx / D4, d0 = (idx % D4) * 4;
    const int m = w.rb * a.rows_pb + rowl;
    if (m >= a.rows) continue;
    const int t = m / a.group, hq = w.kvh * a.group + m % a.group;
    const bool valid = vis[t] != 0ull;
    float mt = kNegInf;
    for (int s = 0; s < w.nsplit; ++s) mt = fmaxf(mt, base[s * pstride + mo + rowl]);
    float lsum = 0.f;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    if (valid && mt != kNegInf) {
      for (int s = 0; s < w.nsplit; ++s) {
        const float* ps = base + s * pstride;
        const float wt = __builtin_amdgcn_exp2f(ps[mo + rowl] - mt);
        lsum += wt * ps[mo + a.rows_pb + rowl];
        acc += wt * *reinterpret_cast<const f32x4*>(ps + rowl * D + d0);
      }
    }
    const bool ok = valid && lsum > 0.f;
    const float inv = ok ? 1.f / lsum : 0.f;
    const int64_t orow = ((static_cast<int64_t>(w.b) * a.n_new + t) * a.hq + hq) * D + d0;
    if constexpr (sizeof(OutT) == 2) {
      u32x2 pk = {pack_bf16x2(acc[0] * inv, acc[1] * inv), pack_bf16x2(acc[2] * inv, acc[3] * inv)};
      *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(a.out) + orow) = pk;
    } else {
      *reinterpret_cast<f32x4*>(static_cast<float*>(a.out) + orow) = acc * inv;
    }
    if (d0 == 0 && a.lse)
      a.lse[(static_cast<int64_t>(w.b) * a.hq + hq) * a.n_new + t] =
          ok ? (mt + __log2f(lsum)) * kLn2 : kNegInf;
  }
}

// Ticket protocol after a partial has been written.  Returns true in the one
// work-group that must merge.  Release fence before the ticket, acquire after.
__device__ inline bool arrive_last(const AttnArgs& a, int64_t pair, int nsplit, int* s_last) {
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) *s_last = (atomicAdd(a.tickets + pair, 1) == nsplit - 1);
  __syncthreads();
  if (!*s_last) return false;
  __threadfence();
  return true;
}

// ----------------------------------------------------------------------------
// bf16 MFMA kernel
// ----------------------------------------------------------------------------
template <int D, int NT, bool PAGED>
__device__ inline void load_kv_tile(uint8_t* sk, uint8_t* sv, const AttnArgs& a, const Work& w,
                                    int k0, bool is_new, int tid) {
  constexpr int CH = D / 8;                  // 16-byte chunks per key row
  constexpr int PER = kTile * CH / NT;       // chunks per thread
  constexpr int ROWB = 2 * D + 16;           // padded LDS row (bytes)
  static_assert(PER >= 1, "tile too small for the work-group");
  u32x4 kr[PER], vr[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int c = tid + i * NT;
    const int row = c / CH, e = (c % CH) * 8;
    const u32x4 zero = {0u, 0u, 0u, 0u};
    kr[i] = zero;
    vr[i] = zero;
    if (is_new) {
      if (row < a.n_new) {
        const int64_t off = ((static_cast<int64_t>(w.b) * a.n_new + row) * a.hkv + w.kvh) * D + e;
        kr[i] = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.k_new) + off);
        vr[i] = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.v_new) + off);
      }
    } else {
      const int key = k0 + row;
      if (key < w.kend) {
        const int64_t off = cache_offset<PAGED>(a, w.b, w.kvh, key, e);
        kr[i] = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.k_cache) + off);
        vr[i] = *reinterpret_cast<const u32x4*>(static_cast<const uint16_t*>(a.v_cache) + off);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int c = tid + i * NT;
    const int row = c / CH, ch = c % CH;
    *reinterpret_cast<u32x4*>(sk + row * ROWB + ch * 16) = kr[i];
    *reinterpret_cast<u32x4*>(sv + row * ROWB + ch * 16) = vr[i];
  }
}

// V^T operands for one 16-key chunk: lane (n, h) supplies keys
// kappa(i) = kbase + 8*(i/4) + 4*h + i%4 (i < 8) at dims DPL*n + c, c < DPL.
template <int D>
__device__ inline void v_operands(const uint8_t* sv, int kbase, int n, int h,
                                  bf16x8 (&va)[D / 32]) {
  constexpr int DPL = D / 32;
  constexpr int ROWB = 2 * D + 16;
  if constexpr (DPL == 4) {
    u32x2 r[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int key = kbase + 8 * (i >> 2) + 4 * h + (i & 3);
      r[i] = *reinterpret_cast<const u32x2*>(sv + key * ROWB + n * 8);
    }
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      u32x4 t;
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        const uint32_t lo = (c < 2) ? r[2 * p][0] : r[2 * p][1];
        const uint32_t hi = (c < 2) ? r[2 * p + 1][0] : r[2 * p + 1][1];
        t[p] = __builtin_amdgcn_perm(hi, lo, (c & 1) ? 0x07060302u : 0x05040100u);
      }
      va[c] = __builtin_bit_cast(bf16x8, t);
    }
  } else {
    uint32_t r[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int key = kbase + 8 * (i >> 2) + 4 * h + (i & 3);
      r[i] = *reinterpret_cast<const uint32_t*>(sv + key * ROWB + n * 4);
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      u32x4 t;
#pragma unroll
      for (int p = 0; p < 4; ++p)
        t[p] = __builtin_amdgcn_perm(r[2 * p + 1], r[2 * p], c ? 0x07060302u : 0x05040100u);
      va[c] = __builtin_bit_cast(bf16x8, t);
    }
  }
}

template <int D, int NW, bool PAGED>
__global__ void __launch_bounds__(NW * 64) attn_bf16_kernel(AttnArgs a) {
  constexpr int NT = NW * 64;
  constexpr int DPL = D / 32;
  constexpr int KS = D / 16;
  constexpr int ROWB = 2 * D + 16;
  __shared__ __attribute__((aligned(16))) uint8_t sk[kTile * ROWB];
  __shared__ __attribute__((aligned(16))) uint8_t sv[kTile * ROWB];
  __shared__ uint64_t vis[kMaxNew];
  __shared__ int s_last;

  Work w;
  if (!setup_work(a, w)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  const int32_t* step_row = a.step_map + static_cast<int64_t>(w.b) * a.B;
  if (tid < kMaxNew)
    vis[tid] = tid < a.n_new ? visibility_word(tid, step_row, w.gamma, a.B, a.n_new) : 0ull;

  const int rowl = wave * 32 + n;
  const int m = w.rb * a.rows_pb + rowl;
  const bool row_in = m < a.rows;
  const int t = row_in ? m / a.group : 0;
  const int hq = w.kvh * a.group + (row_in ? m % a.group : 0);

  // Q^T operands of this lane's row: dims 16*ks + 8*h + [0, 8).
  bf16x8 qop[KS];
  {
    const bf16x8* qrow = reinterpret_cast<const bf16x8*>(
        static_cast<const uint16_t*>(a.q) + ((static_cast<int64_t>(w.b) * a.n_new + t) * a.hq + hq) * D);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (row_in) {
        qop[ks] = qrow[2 * ks + h];
      } else {
        const u32x4 z = {0u, 0u, 0u, 0u};
        qop[ks] = __builtin_bit_cast(bf16x8, z);
      }
    }
  }
  __syncthreads();
  const uint64_t myvis = row_in ? vis[t] : 0ull;

  f32x16 o[DPL];
#pragma unroll
  for (int c = 0; c < DPL; ++c)
#pragma unroll
    for (int j = 0; j < 16; ++j) o[c][j] = 0.f;
  float m_run = kNegInf, l_run = 0.f;
  const float sl2 = a.scale_log2;

  const int ntp = w.kend > w.kbeg ? (w.kend - w.kbeg + kTile - 1) / kTile : 0;
  const int nt = ntp + (w.split == 0 ? 1 : 0);
  for (int it = 0; it < nt; ++it) {
    const bool is_new = it == ntp;
    const int k0 = w.kbeg + it * kTile;
    if (it > 0) __syncthreads();
    load_kv_tile<D, NT, PAGED>(sk, sv, a, w, k0, is_new, tid);
    __syncthreads();

    // S^T = K Q^T: two 32-key blocks.  Register j of block kb holds key
    // 32*kb + 8*(j/4) + 4*h + j%4 of this lane's row.
    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int j = 0; j < 16; ++j) s[kb][j] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 ka =
            *reinterpret_cast<const bf16x8*>(sk + (32 * kb + n) * ROWB + (16 * ks + 8 * h) * 2);
        s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qop[ks], s[kb], 0, 0, 0);
      }
    }
    if (is_new) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int key = 32 * kb + 8 * (j >> 2) + 4 * h + (j & 3);
          if (!((myvis >> key) & 1ull)) s[kb][j] = kNegInf;
        }
    } else if (k0 + kTile > w.kend) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int key = k0 + 32 * kb + 8 * (j >> 2) + 4 * h + (j & 3);
          if (key >= w.kend) s[kb][j] = kNegInf;
        }
    }

    float mx = kNegInf;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int j = 0; j < 16; ++j) mx = fmaxf(mx, s[kb][j]);
    mx = fmaxf(mx, __shfl_xor(mx, 32));
    const float m_new = fmaxf(m_run, mx * sl2);
    if (m_new > m_run + kLazy) {
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      l_run *= alpha;
#pragma unroll
      for (int c = 0; c < DPL; ++c) o[c] *= alpha;
      m_run = m_new;
    }
    const float moff = m_run == kNegInf ? 0.f : m_run;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[kb][j], sl2, -moff));
        s[kb][j] = p;
        l_run += p;
      }

    // O^T += V^T P^T, one 16-key chunk at a time.
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        u32x4 pw;
#pragma unroll
        for (int p = 0; p < 4; ++p) pw[p] = pack_bf16x2(s[kb][8 * hf + 2 * p], s[kb][8 * hf + 2 * p + 1]);
        const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
        bf16x8 va[DPL];
        v_operands<D>(sv, 32 * kb + 16 * hf, n, h, va);
#pragma unroll
        for (int c = 0; c < DPL; ++c)
          o[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va[c], pb, o[c], 0, 0, 0);
      }
  }
  const float l_tot = l_run + __shfl_xor(l_run, 32);

  // Register j of o[c] holds dim DPL*(8*(j/4) + 4*h + j%4) + c of this row.
  if (w.nsplit == 1) {
    if (!row_in) return;
    const bool valid = myvis != 0ull;
    const float inv = valid ? 1.f / l_tot : 0.f;
    uint16_t* orow = static_cast<uint16_t*>(a.out) +
                     ((static_cast<int64_t>(w.b) * a.n_new + t) * a.hq + hq) * D;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if constexpr (DPL == 4) {
        u32x4 lo, hi;
#pragma unroll
        for (int jj = 0; jj < 2; ++jj) {
          lo[2 * jj] = pack_bf16x2(o[0][4 * q + jj] * inv, o[1][4 * q + jj] * inv);
          lo[2 * jj + 1] = pack_bf16x2(o[2][4 * q + jj] * inv, o[3][4 * q + jj] * inv);
          hi[2 * jj] = pack_bf16x2(o[0][4 * q + 2 + jj] * inv, o[1][4 * q + 2 + jj] * inv);
          hi[2 * jj + 1] = pack_bf16x2(o[2][4 * q + 2 + jj] * inv, o[3][4 * q + 2 + jj] * inv);
        }
        *reinterpret_cast<u32x4*>(orow + 32 * q + 16 * h) = lo;
        *reinterpret_cast<u32x4*>(orow + 32 * q + 16 * h + 8) = hi;
      } else {
        u32x4 v;
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) v[jj] = pack_bf16x2(o[0][4 * q + jj] * inv, o[1][4 * q + jj] * inv);
        *reinterpret_cast<u32x4*>(orow + 16 * q + 8 * h) = v;
      }
    }
    if (a.lse && h == 0)
      a.lse[(static_cast<int64_t>(w.b) * a.hq + hq) * a.n_new + t] =
          valid ? (m_run + __log2f(l_tot)) * kLn2 : kNegInf;
    return;
  }

  const int64_t pair = (static_cast<int64_t>(w.b) * a.hkv + w.kvh) * a.row_blocks + w.rb;
  float* part = a.part + (pair * a.splits + w.split) * static_cast<int64_t>(a.rows_pb) * (D + 2);
  if (row_in) {
    float* prow = part + rowl * D;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        if constexpr (DPL == 4) {
          const f32x4 v = {o[0][4 * q + jj], o[1][4 * q + jj], o[2][4 * q + jj], o[3][4 * q + jj]};
          *reinterpret_cast<f32x4*>(prow + 32 * q + 16 * h + 4 * jj) = v;
        } else if (jj % 2 == 0) {
          const f32x4 v = {o[0][4 * q + jj], o[1][4 * q + jj], o[0][4 * q + jj + 1], o[1][4 * q + jj + 1]};
          *reinterpret_cast<f32x4*>(prow + 16 * q + 8 * h + 2 * jj) = v;
        }
      }
    }
    if (h == 0) {
      part[a.rows_pb * D + rowl] = m_run;
      part[a.rows_pb * D + a.rows_pb + rowl] = l_tot;
    }
  }
  if (!arrive_last(a, pair, w.nsplit, &s_last)) return;
  merge_splits<D, NT, uint16_t>(a, pair, w, vis, tid);
  if (tid == 0) atomicExch(a.tickets + pair, 0);
}

// ----------------------------------------------------------------------------
// float32 kernel (VALU).  A wave works on one row at a time (8 rows per wave,
// 32 rows per work-group); the running output, max and sum of each row live
// in LDS.  For a 16-key tile, lanes 16*q + j (q < 4) each take a quarter of
// the dot product of key j; lanes own dims lane + 64*u of the output.
// ----------------------------------------------------------------------------
template <int D, bool PAGED>
__global__ void __launch_bounds__(256) attn_f32_kernel(AttnArgs a) {
  constexpr int NT = 256, TK = 16, RPW = 8, KROW = D + 1, DU = D / 64, QD = D / 4;
  __shared__ float sk[TK * KROW];
  __shared__ float sv[TK * D];
  __shared__ float sq[32 * D];
  __shared__ float so[32 * D];
  __shared__ float sm[32], sl[32];
  __shared__ uint64_t vis[kMaxNew];
  __shared__ int s_last;

  Work w;
  if (!setup_work(a, w)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t* step_row = a.step_map + static_cast<int64_t>(w.b) * a.B;
  if (tid < kMaxNew)
    vis[tid] = tid < a.n_new ? visibility_word(tid, step_row, w.gamma, a.B, a.n_new) : 0ull;
  if (tid < 32) {
    sm[tid] = kNegInf;
    sl[tid] = 0.f;
  }
  for (int idx = tid; idx < 32 * D; idx += NT) {
    const int rowl = idx / D, d = idx % D;
    const int m = w.rb * a.rows_pb + rowl;
    float v = 0.f;
    if (m < a.rows) {
      const int t = m / a.group, hq = w.kvh * a.group + m % a.group;
      v = static_cast<const float*>(a.q)[((static_cast<int64_t>(w.b) * a.n_new + t) * a.hq + hq) * D + d];
    }
    sq[idx] = v;
    so[idx] = 0.f;
  }

  const float sl2 = a.scale_log2;
  const int ntp = w.kend > w.kbeg ? (w.kend - w.kbeg + TK - 1) / TK : 0;
  const int ntn = w.split == 0 ? (a.n_new + TK - 1) / TK : 0;
  const int j = lane & 15, qtr = lane >> 4;
  for (int it = 0; it < ntp + ntn; ++it) {
    const bool is_new = it >= ntp;
    const int k0 = is_new ? (it - ntp) * TK : w.kbeg + it * TK;
    __syncthreads();
    for (int idx = tid; idx < TK * D; idx += NT) {
      const int row = idx / D, e = idx % D;
      float kv = 0.f, vv = 0.f;
      if (is_new) {
        const int slot = k0 + row;
        if (slot < a.n_new) {
          const int64_t off = ((static_cast<int64_t>(w.b) * a.n_new + slot) * a.hkv + w.kvh) * D + e;
          kv = static_cast<const float*>(a.k_new)[off];
          vv = static_cast<const float*>(a.v_new)[off];
        }
      } else if (k0 + row < w.kend) {
        const int64_t off = cache_offset<PAGED>(a, w.b, w.kvh, k0 + row, e);
        kv = static_cast<const float*>(a.k_cache)[off];
        vv = static_cast<const float*>(a.v_cache)[off];
      }
      sk[row * KROW + e] = kv;
      sv[row * D + e] = vv;
    }
    __syncthreads();
    for (int r = 0; r < RPW; ++r) {
      const int rowl = wave * RPW + r;
      const int m = w.rb * a.rows_pb + rowl;
      const uint64_t rv = m < a.rows ? vis[m / a.group] : 0ull;
      float s = 0.f;
      for (int d = 0; d < QD; ++d) s = fmaf(sq[rowl * D + qtr * QD + d], sk[j * KROW + qtr * QD + d], s);
      s += __shfl_xor(s, 16);
      s += __shfl_xor(s, 32);
      const bool ok = is_new ? ((rv >> (k0 + j)) & 1ull) != 0ull : (k0 + j < w.kend);
      s = ok ? s * sl2 : kNegInf;
      float mx = s;
#pragma unroll
      for (int sh = 8; sh >= 1; sh >>= 1) mx = fmaxf(mx, __shfl_xor(mx, sh));
      const float m_old = sm[rowl];
      const float m_new = fmaxf(m_old, mx);
      const float moff = m_new == kNegInf ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_old - moff);
      const float p = __builtin_amdgcn_exp2f(s - moff);
      float ps = p;
#pragma unroll
      for (int sh = 8; sh >= 1; sh >>= 1) ps += __shfl_xor(ps, sh);
      float acc[DU];
#pragma unroll
      for (int u = 0; u < DU; ++u) acc[u] = so[rowl * D + lane + 64 * u] * alpha;
      for (int jj = 0; jj < TK; ++jj) {
        const float pj = __shfl(p, jj);
#pragma unroll
        for (int u = 0; u < DU; ++u) acc[u] = fmaf(pj, sv[jj * D + lane + 64 * u], acc[u]);
      }
#pragma unroll
      for (int u = 0; u < DU; ++u) so[rowl * D + lane + 64 * u] = acc[u];
      if (lane == 0) {
        sl[rowl] = sl[rowl] * alpha + ps;
        sm[rowl] = m_new;
      }
    }
  }
  __syncthreads();

  if (w.nsplit == 1) {
    for (int r = 0; r < RPW; ++r) {
      const int rowl = wave * RPW + r;
      const int m = w.rb * a.rows_pb + rowl;
      if (m >= a.rows) continue;
      const int t = m / a.group, hq = w.kvh * a.group + m % a.group;
      const bool valid = vis[t] != 0ull;
      const float inv = valid ? 1.f / sl[rowl] : 0.f;
      float* orow = static_cast<float*>(a.out) + ((static_cast<int64_t>(w.b) * a.n_new + t) * a.hq + hq) * D;
#pragma unroll
      for (int u = 0; u < DU; ++u) orow[lane + 64 * u] = so[rowl * D + lane + 64 * u] * inv;
      if (a.lse && lane == 0)
        a.lse[(static_cast<int64_t>(w.b) * a.hq + hq) * a.n_new + t] =
            valid ? (sm[rowl] + __log2f(sl[rowl])) * kLn2 : kNegInf;
    }
    return;
  }
  const int64_t pair = (static_cast<int64_t>(w.b) * a.hkv + w.kvh) * a.row_blocks + w.rb;
  float* part = a.part + (pair * a.splits + w.split) * static_cast<int64_t>(a.rows_pb) * (D + 2);
  for (int idx = tid; idx < 32 * D; idx += NT) part[idx] = so[idx];
  if (tid < 32) {
    part[a.rows_pb * D + tid] = sm[tid];
    part[a.rows_pb * D + a.rows_pb + tid] = sl[tid];
  }
  if (!arrive_last(a, pair, w.nsplit, &s_last)) return;
  merge_splits<D, NT, float>(a, pair, w, vis, tid);
  if (tid == 0) atomicExch(a.tickets + pair, 0);
}

template <int D, bool PAGED>
hipError_t launch_bf16(int waves, dim3 grid, const AttnArgs& a, hipStream_t st) {
  switch (waves) {
    case 1: hipLaunchKernelGGL((attn_bf16_kernel<D, 1, PAGED>), grid, dim3(64), 0, st, a); break;
    case 2: hipLaunchKernelGGL((attn_bf16_kernel<D, 2, PAGED>), grid, dim3(128), 0, st, a); break;
    case 4: hipLaunchKernelGGL((attn_bf16_kernel<D, 4, PAGED>), grid, dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL((attn_bf16_kernel<D, 8, PAGED>), grid, dim3(512), 0, st, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention(const simsd_attn_desc& d, const AttnPlan& p, const AttnArgs& a,
                            hipStream_t st) {
  const dim3 grid(p.splits, d.num_kv_heads * p.row_blocks, d.batch);
  const bool paged = d.page_size > 0;
  if (d.dtype == SIMSD_BF16) {
    if (d.head_dim == 128)
      return paged ? launch_bf16<128, true>(p.waves, grid, a, st)
                   : launch_bf16<128, false>(p.waves, grid, a, st);
    return paged ? launch_bf16<64, true>(p.waves, grid, a, st)
                 : launch_bf16<64, false>(p.waves, grid, a, st);
  }
  if (d.head_dim == 128) {
    if (paged) hipLaunchKernelGGL((attn_f32_kernel<128, true>), grid, dim3(256), 0, st, a);
    else hipLaunchKernelGGL((attn_f32_kernel<128, false>), grid, dim3(256), 0, st, a);
  } else {
    if (paged) hipLaunchKernelGGL((attn_f32_kernel<64, true>), grid, dim3(256), 0, st, a);
    else hipLaunchKernelGGL((attn_f32_kernel<64, false>), grid, dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

}  // namespace simsd
