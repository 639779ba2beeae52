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
// into the rows of one row block (GQA packing), so each K/V byte of the prefix
// is read from HBM once per KV head.  When a sequence's prefix spans several
// chunks, each chunk writes an unnormalised partial output with its running
// max and sum, and a second kernel merges them; there is no device-wide fence
// or counter in the streaming kernel.
//
// bf16 path: K and V tiles of 64 keys are loaded into registers one tile ahead
// (two ahead for 8-wave groups) and written to a double-buffered LDS ring with
// 288-byte rows (no bank conflicts for the reads below).  Scores are computed
// transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16, so lane l owns query
// row l % 32 of its wave's 32-row block and a row's softmax state stays in two
// lanes (l, l ^ 32).  O^T = V^T P^T takes P straight from the score registers
// as the B operand; the V^T operand comes from LDS transpose reads
// (ds_read_b64_tr_b16), so no register shuffles are needed.  Row maxima are
// kept in log2 units and rescaled only when they grow by more than 2^8.
#include "simsd_kernels.h"

namespace simsd {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
#define SIMSD_LDS __attribute__((address_space(3)))

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


// Which prefix keys a work-group owns.
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

// Partial layout per (pair, split): O[rows_pb][D] (unnormalised, fp32), then
// m[rows_pb] (log2 units), then l[rows_pb].
__device__ inline float* partial_base(const AttnArgs& a, const Work& w, int D) {
  const int64_t pair = (static_cast<int64_t>(w.b) * a.hkv + w.kvh) * a.row_blocks + w.rb;
  return a.part + (pair * a.splits + w.split) * static_cast<int64_t>(a.rows_pb) * (D + 2);
}

// ----------------------------------------------------------------------------
// bf16 MFMA kernel
// ----------------------------------------------------------------------------
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two floats -> two bf16 (round to nearest even) in one instruction.
__device__ inline uint32_t pack2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

template <int D>
struct TileGeom {
  static constexpr int CH = D / 8;             // 16-byte chunks per key row
  static constexpr int ROWB = 2 * D;           // LDS bytes per key row (unpadded)
  static constexpr int TILEB = kTile * ROWB;   // one tensor (K or V) of one tile
};

// LDS swizzle: 16-byte chunk L of key row r is stored at chunk L ^ swz(r).  The
// XOR masks were chosen (by exhaustive search over linear maps of r mod 16) so
// that the K operand reads (32 rows, one chunk) and the transpose reads of V
// (4 rows x 4 chunks per 32 lanes) hit distinct banks with 32 or 64 LDS banks.
template <int D>
__device__ inline int swz(int r) {
  if constexpr (D == 128)
    return ((r & 1) ? 4 : 0) ^ ((r & 2) ? 10 : 0) ^ ((r & 4) ? 1 : 0) ^ ((r & 8) ? 2 : 0);
  else
    return ((r & 1) ? 2 : 0) ^ ((r & 2) ? 4 : 0) ^ ((r & 4) ? 1 : 0) ^ ((r & 8) ? 2 : 0);
}

constexpr int kMaxChunkPages = 512;            // page ids of one chunk staged in LDS

// Streams 64-key K/V tiles of one work-group's chunk into registers.  A thread
// owns chunks c = tid + i*NT of a tile: key rows row0 + i*RSTEP, elements
// [e0, e0 + 8).  Full prefix tiles load unguarded from a per-tile base plus a
// per-thread constant offset; the tail tile and the new-slot tile are guarded.
template <int D, int NT, bool PAGED>
struct KVStream {
  static constexpr int CH = TileGeom<D>::CH;
  static constexpr int PER = kTile * CH / NT;
  static constexpr int RSTEP = NT / CH;
  static_assert(PER >= 1 && NT % CH == 0, "tile too small for the work-group");

  const char* kc;        // k_cache (bytes)
  const char* vc;        // v_cache
  int64_t seqoff;        // contiguous: sequence offset (bytes)
  int64_t tokb, pageb;   // bytes per token / per page (paged)
  int64_t toff;          // contiguous: (row0 * tok + kvh * head + e0) bytes; paged: (kvh * head + e0) bytes
  int row0, e0, P;
  bool lds_pages;        // page ids of this chunk are staged in s_pg
  int pg_first;          // first page index of the chunk (in the sequence's block table)
  const int32_t* bt;     // this sequence's block table row

  __device__ inline void init(const AttnArgs& a, const Work& w, int tid, int* s_pg) {
    row0 = tid / CH;
    e0 = (tid % CH) * 8;
    kc = static_cast<const char*>(a.k_cache);
    vc = static_cast<const char*>(a.v_cache);
    tokb = a.cs_tok * 2;
    const int64_t hoff = (static_cast<int64_t>(w.kvh) * a.cs_head + e0) * 2;
    if (PAGED) {
      P = a.page_size;
      pageb = a.cs_seq * 2;
      toff = hoff;
      bt = a.block_table + static_cast<int64_t>(w.b) * a.max_pages;
      pg_first = w.kbeg / P;
      const int npg = w.kend > w.kbeg ? (w.kend - 1) / P - pg_first + 1 : 0;
      lds_pages = (kTile % P == 0) && npg <= kMaxChunkPages;
      if (lds_pages)
        for (int j = tid; j < npg; j += NT) s_pg[j] = bt[pg_first + j];
    } else {
      seqoff = static_cast<int64_t>(w.b) * a.cs_seq * 2;
      toff = static_cast<int64_t>(row0) * tokb + hoff;
    }
  }

  // Byte offset of this thread's chunk i of the prefix tile starting at key k0.
  __device__ inline int64_t offset(int k0, int i, const int* s_pg) const {
    const int row = row0 + i * RSTEP;
    if (!PAGED) return seqoff + static_cast<int64_t>(k0 + i * RSTEP) * tokb + toff;
    int64_t page;
    int in_page;
    if (lds_pages) {                          // P divides the tile: k0 % P == 0
      page = s_pg[(k0 / P - pg_first) + row / P];
      in_page = row % P;
    } else {
      const int key = k0 + row;
      page = bt[key / P];
      in_page = key % P;
    }
    return page * pageb + static_cast<int64_t>(in_page) * tokb + toff;
  }

  __device__ inline void load(u32x4 (&k)[PER], u32x4 (&v)[PER], const AttnArgs& a, const Work& w,
                              int k0, bool is_new, const int* s_pg) const {
    const u32x4 zero = {0u, 0u, 0u, 0u};
    if (is_new) {
      const char* kn = static_cast<const char*>(a.k_new);
      const char* vn = static_cast<const char*>(a.v_new);
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int row = row0 + i * RSTEP;
        k[i] = zero;
        v[i] = zero;
        if (row < a.n_new) {
          const int64_t off = (((static_cast<int64_t>(w.b) * a.n_new + row) * a.hkv + w.kvh) * D + e0) * 2;
          k[i] = *reinterpret_cast<const u32x4*>(kn + off);
          v[i] = *reinterpret_cast<const u32x4*>(vn + off);
        }
      }
    } else if (k0 + kTile <= w.kend) {
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const int64_t off = offset(k0, i, s_pg);
        k[i] = *reinterpret_cast<const u32x4*>(kc + off);
        v[i] = *reinterpret_cast<const u32x4*>(vc + off);
      }
    } else {
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        k[i] = zero;
        v[i] = zero;
        if (k0 + row0 + i * RSTEP < w.kend) {
          const int64_t off = offset(k0, i, s_pg);
          k[i] = *reinterpret_cast<const u32x4*>(kc + off);
          v[i] = *reinterpret_cast<const u32x4*>(vc + off);
        }
      }
    }
  }

  __device__ inline void store(uint8_t* sk, uint8_t* sv, const u32x4 (&k)[PER],
                               const u32x4 (&v)[PER]) const {
    constexpr int ROWB = TileGeom<D>::ROWB;
#pragma unroll
    for (int i = 0; i < PER; ++i) {
      const int row = row0 + i * RSTEP;
      const int off = row * ROWB + 16 * ((e0 / 8) ^ swz<D>(row));
      *reinterpret_cast<u32x4*>(sk + off) = k[i];
      *reinterpret_cast<u32x4*>(sv + off) = v[i];
    }
  }
};

// RW row waves of 32 rows each; KW = 2 pairs every row wave with a second wave
// that takes the other 32-key half of each tile (small row blocks, where the
// extra wave doubles the loads in flight); the two halves merge at the end.
template <int D, int RW, int KW, bool PAGED>
__global__ void __launch_bounds__(RW * KW * 64, 2) attn_bf16_kernel(AttnArgs a) {
  constexpr int NW = RW * KW;
  constexpr int NT = NW * 64;
  constexpr int NB = D / 32;                   // 32-dim output blocks
  constexpr int KS = D / 16;                   // k-steps of QK^T
  constexpr int ROWB = TileGeom<D>::ROWB;
  constexpr int TILEB = TileGeom<D>::TILEB;
  constexpr int PF = NW >= 8 ? 2 : 1;          // tiles prefetched into registers
  using Stream = KVStream<D, NT, PAGED>;
  constexpr int PER = Stream::PER;
  __shared__ __attribute__((aligned(16))) uint8_t smem[2][2][TILEB];   // [buffer][K, V]
  __shared__ uint64_t vis[kMaxNew];
  __shared__ int s_pg[PAGED ? kMaxChunkPages : 1];

  Work w;
  if (!setup_work(a, w)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = lane & 31, h = lane >> 5;
  const int rw = wave % RW, kw = wave / RW;    // row wave, key half

  const int rowl = rw * 32 + n;
  const int m = w.rb * a.rows_pb + rowl;
  const bool row_in = m < a.rows;
  const int t = row_in ? m / a.group : 0;
  const int hq = w.kvh * a.group + (row_in ? m % a.group : 0);

  // Q^T operands of this lane's row (dims 16*ks + 8*h + [0, 8)), loaded first
  // so that they have landed before the tile loop starts.
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
  const int32_t* step_row = a.step_map + static_cast<int64_t>(w.b) * a.B;
  if (tid < kMaxNew)
    vis[tid] = tid < a.n_new ? visibility_word(tid, step_row, w.gamma, a.B, a.n_new) : 0ull;

  Stream kv;
  kv.init(a, w, tid, s_pg);
  if (PAGED) __syncthreads();                  // staged page ids

  const int ntp = w.kend > w.kbeg ? (w.kend - w.kbeg + kTile - 1) / kTile : 0;
  const int nt = ntp + (w.split == 0 ? 1 : 0);
  auto tile_k0 = [&](int it) { return w.kbeg + it * kTile; };

  u32x4 rk[PF][PER], rv[PF][PER];
  kv.load(rk[0], rv[0], a, w, tile_k0(0), 0 == ntp, s_pg);
  kv.store(smem[0][0], smem[0][1], rk[0], rv[0]);
#pragma unroll
  for (int p = 0; p < PF; ++p)
    if (1 + p < nt) kv.load(rk[(1 + p) % PF], rv[(1 + p) % PF], a, w, tile_k0(1 + p), 1 + p == ntp, s_pg);
  __syncthreads();
  const uint64_t myvis = row_in ? vis[t] : 0ull;

  f32x16 o[NB];
#pragma unroll
  for (int c = 0; c < NB; ++c)
#pragma unroll
    for (int j = 0; j < 16; ++j) o[c][j] = 0.f;
  float m_run = kNegInf, l_run = 0.f;
  const float sl2 = a.scale_log2;

  // Per-lane LDS read offsets (swizzled).  K operand of k-step ks: row n of a
  // 32-key block, chunk 2*ks + h.  V transpose reads: lane (g = lane/16,
  // k = (lane%16)/4, q = lane%4) reads 4 dims at column 32*c + 16*(g%2) + 4*q
  // of key row 4*h + k (lo) or 8 + 4*h + k (hi) of a 16-key chunk.
  int koff[KS], voff[NB][2];
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) koff[ks] = n * ROWB + 16 * ((2 * ks + h) ^ swz<D>(n));
  {
    const int k = (lane & 15) >> 2, q = lane & 3, gg = (lane >> 4) & 1;
#pragma unroll
    for (int c = 0; c < NB; ++c)
#pragma unroll
      for (int hl = 0; hl < 2; ++hl) {
        const int r = 8 * hl + 4 * h + k;
        const int L = 4 * c + 2 * gg + (q >> 1);
        voff[c][hl] = r * ROWB + 16 * (L ^ swz<D>(r)) + 8 * (q & 1);
      }
  }

  // The loop is unrolled by two: the LDS buffer and the register set are then
  // compile-time indices (a runtime index would put the sets in scratch).
  for (int it0 = 0; it0 < nt; it0 += 2) {
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    const int it = it0 + u;
    if (it >= nt) break;
    const bool is_new = it == ntp;
    const int k0 = tile_k0(it);
    const uint8_t* sk = smem[u][0];
    const uint8_t* sv = smem[u][1];

#pragma unroll
    for (int kb0 = 0; kb0 < 2 / KW; ++kb0) {
      const int kb = KW == 1 ? kb0 : kw;
      // S^T = K Q^T for one 32-key block.  Register j holds key
      // 32*kb + 8*(j/4) + 4*h + j%4 of this lane's row.
      f32x16 s;
#pragma unroll
      for (int j = 0; j < 16; ++j) s[j] = 0.f;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const bf16x8 ka = *reinterpret_cast<const bf16x8*>(sk + 32 * kb * ROWB + koff[ks]);
        s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qop[ks], s, 0, 0, 0);
      }
      if (is_new) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int key = 32 * kb + 8 * (j >> 2) + 4 * h + (j & 3);
          if (!((myvis >> key) & 1ull)) s[j] = kNegInf;
        }
      } else if (k0 + kTile > w.kend) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int key = k0 + 32 * kb + 8 * (j >> 2) + 4 * h + (j & 3);
          if (key >= w.kend) s[j] = kNegInf;
        }
      }

      float mx = kNegInf;
#pragma unroll
      for (int j = 0; j < 16; ++j) mx = fmaxf(mx, s[j]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx * sl2);
      if (m_new > m_run + kLazy) {
        const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
        l_run *= alpha;
#pragma unroll
        for (int c = 0; c < NB; ++c) o[c] *= alpha;
        m_run = m_new;
      }
      const float moff = m_run == kNegInf ? 0.f : m_run;
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[j], sl2, -moff));
        s[j] = p;
        l_run += p;
      }

      // O^T += V^T P^T, two 16-key chunks.  Chunk hf covers keys
      // 32*kb + 16*hf + kappa(h, i), kappa(h, i) = 8*(i/4) + 4*h + i%4.
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        u32x4 pw;
#pragma unroll
        for (int p = 0; p < 4; ++p) pw[p] = pack2(s[8 * hf + 2 * p], s[8 * hf + 2 * p + 1]);
        const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
        const uint8_t* vblk = sv + (32 * kb + 16 * hf) * ROWB;
#pragma unroll
        for (int c = 0; c < NB; ++c) {
          const s16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((SIMSD_LDS s16x4*)(vblk + voff[c][0]));
          const s16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((SIMSD_LDS s16x4*)(vblk + voff[c][1]));
          const u32x2 l2 = __builtin_bit_cast(u32x2, lo), h2 = __builtin_bit_cast(u32x2, hi);
          const u32x4 vw = {l2[0], l2[1], h2[0], h2[1]};
          o[c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, vw), pb, o[c], 0, 0, 0);
        }
      }
    }

    // Next tile: registers -> the other LDS buffer, then refill the registers.
    if (it + 1 < nt) {
      const int nx = (u + 1) % PF;         // a constant once the u loop is unrolled
      kv.store(smem[1 - u][0], smem[1 - u][1], rk[nx], rv[nx]);
      if (it + 1 + PF < nt)
        kv.load(rk[nx], rv[nx], a, w, tile_k0(it + 1 + PF), it + 1 + PF == ntp, s_pg);
    }
    __syncthreads();
  }
  }
  if constexpr (KW == 2) {
    // Merge the two key halves of each row through LDS (the tiles are free).
    constexpr int SLOT = NB * 16 + 2;
    float* xs = reinterpret_cast<float*>(&smem[0][0][0]) + (rw * 64 + lane) * SLOT;
    if (kw == 1) {
#pragma unroll
      for (int c = 0; c < NB; ++c)
#pragma unroll
        for (int j = 0; j < 16; ++j) xs[c * 16 + j] = o[c][j];
      xs[NB * 16] = m_run;
      xs[NB * 16 + 1] = l_run;
    }
    __syncthreads();
    if (kw == 1) return;
    const float m1 = xs[NB * 16], l1 = xs[NB * 16 + 1];
    const float mm = fmaxf(m_run, m1);
    const float mref = mm == kNegInf ? 0.f : mm;
    const float a0 = __builtin_amdgcn_exp2f(m_run - mref), a1 = __builtin_amdgcn_exp2f(m1 - mref);
#pragma unroll
    for (int c = 0; c < NB; ++c)
#pragma unroll
      for (int j = 0; j < 16; ++j) o[c][j] = o[c][j] * a0 + xs[c * 16 + j] * a1;
    l_run = l_run * a0 + l1 * a1;
    m_run = mm;
  }
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  if (!row_in) return;

  // Register j of o[c] holds dim 32*c + 8*(j/4) + 4*h + j%4 of this row.
  if (w.nsplit == 1) {
    const bool valid = myvis != 0ull;
    const float inv = valid ? 1.f / l_tot : 0.f;
    uint16_t* orow = static_cast<uint16_t*>(a.out) +
                     ((static_cast<int64_t>(w.b) * a.n_new + t) * a.hq + hq) * D;
#pragma unroll
    for (int c = 0; c < NB; ++c)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const u32x2 v = {pack2(o[c][4 * q] * inv, o[c][4 * q + 1] * inv),
                         pack2(o[c][4 * q + 2] * inv, o[c][4 * q + 3] * inv)};
        *reinterpret_cast<u32x2*>(orow + 32 * c + 8 * q + 4 * h) = v;
      }
    if (a.lse && h == 0)
      a.lse[(static_cast<int64_t>(w.b) * a.hq + hq) * a.n_new + t] =
          valid ? (m_run + __log2f(l_tot)) * kLn2 : kNegInf;
    return;
  }
  float* part = partial_base(a, w, D);
  float* prow = part + rowl * D;
#pragma unroll
  for (int c = 0; c < NB; ++c)
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const f32x4 v = {o[c][4 * q], o[c][4 * q + 1], o[c][4 * q + 2], o[c][4 * q + 3]};
      *reinterpret_cast<f32x4*>(prow + 32 * c + 8 * q + 4 * h) = v;
    }
  if (h == 0) {
    part[a.rows_pb * D + rowl] = m_run;
    part[a.rows_pb * D + a.rows_pb + rowl] = l_tot;
  }
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
  float* part = partial_base(a, w, D);
  for (int idx = tid; idx < 32 * D; idx += NT) part[idx] = so[idx];
  if (tid < 32) {
    part[a.rows_pb * D + tid] = sm[tid];
    part[a.rows_pb * D + a.rows_pb + tid] = sl[tid];
  }
}

// ----------------------------------------------------------------------------
// Merge of split partials.  Grid: (32-row groups of a row block, KV head x row
// block, sequence); one thread per (row, 4 dims).  Sequences whose prefix fits
// one chunk were finished by the attention kernel and are skipped.
// ----------------------------------------------------------------------------
template <int D, typename OutT>
__global__ void __launch_bounds__(256) merge_kernel(AttnArgs a) {
  constexpr int D4 = D / 4;
  const int b = blockIdx.z;
  const int kvh = blockIdx.y / a.row_blocks, rb = blockIdx.y % a.row_blocks;
  const int plen = min(max(a.prefix_lens[b], 0), a.max_prefix);
  const int nsplit = plen > 0 ? (plen + a.chunk - 1) / a.chunk : 1;
  if (nsplit <= 1) return;
  const int idx = blockIdx.x * 256 + threadIdx.x;
  const int rowl = idx / D4, d0 = (idx % D4) * 4;
  if (rowl >= a.rows_pb) return;
  const int m = rb * a.rows_pb + rowl;
  if (m >= a.rows) return;
  const int t = m / a.group, hq = kvh * a.group + m % a.group;
  const int gamma = min(max(a.num_ref[b], 0), a.L);
  // A row is padding iff it sees no new slot (a non-padded row always sees itself).
  bool valid;
  if (t < a.B) valid = a.step_map[static_cast<int64_t>(b) * a.B + t] >= 0;
  else valid = (t - a.B) < gamma;

  const int64_t pair = (static_cast<int64_t>(b) * a.hkv + kvh) * a.row_blocks + rb;
  const int64_t pstride = static_cast<int64_t>(a.rows_pb) * (D + 2);
  const float* base = a.part + pair * a.splits * pstride;
  const int mo = a.rows_pb * D;
  float mt = kNegInf;
  for (int s = 0; s < nsplit; ++s) mt = fmaxf(mt, base[s * pstride + mo + rowl]);
  float lsum = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  if (valid && mt != kNegInf) {
#pragma unroll 4
    for (int s = 0; s < nsplit; ++s) {
      const float* ps = base + s * pstride;
      const float wt = __builtin_amdgcn_exp2f(ps[mo + rowl] - mt);
      lsum += wt * ps[mo + a.rows_pb + rowl];
      acc += wt * *reinterpret_cast<const f32x4*>(ps + rowl * D + d0);
    }
  }
  const bool ok = valid && lsum > 0.f;
  const float inv = ok ? 1.f / lsum : 0.f;
  const int64_t orow = ((static_cast<int64_t>(b) * a.n_new + t) * a.hq + hq) * D + d0;
  if constexpr (sizeof(OutT) == 2) {
    const u32x2 pk = {pack2(acc[0] * inv, acc[1] * inv), pack2(acc[2] * inv, acc[3] * inv)};
    *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(a.out) + orow) = pk;
  } else {
    *reinterpret_cast<f32x4*>(static_cast<float*>(a.out) + orow) = acc * inv;
  }
  if (d0 == 0 && a.lse)
    a.lse[(static_cast<int64_t>(b) * a.hq + hq) * a.n_new + t] =
        ok ? (mt + __log2f(lsum)) * kLn2 : kNegInf;
}

template <int D, bool PAGED>
void launch_bf16(int row_waves, dim3 grid, const AttnArgs& a, hipStream_t st) {
  switch (row_waves) {
    case 2: hipLaunchKernelGGL((attn_bf16_kernel<D, 2, 2, PAGED>), grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((attn_bf16_kernel<D, 4, 1, PAGED>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((attn_bf16_kernel<D, 8, 1, PAGED>), grid, dim3(512), 0, st, a); break;
  }
}

template <int D>
void launch_f32(bool paged, dim3 grid, const AttnArgs& a, hipStream_t st) {
  if (paged) hipLaunchKernelGGL((attn_f32_kernel<D, true>), grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL((attn_f32_kernel<D, false>), grid, dim3(256), 0, st, a);
}

}  // namespace

hipError_t launch_attention(const simsd_attn_desc& d, const AttnPlan& p, const AttnArgs& a,
                            hipStream_t st) {
  const dim3 grid(p.splits, d.num_kv_heads * p.row_blocks, d.batch);
  const bool paged = d.page_size > 0;
  if (d.dtype == SIMSD_BF16) {
    if (d.head_dim == 128) {
      if (paged) launch_bf16<128, true>(p.row_waves, grid, a, st);
      else launch_bf16<128, false>(p.row_waves, grid, a, st);
    } else {
      if (paged) launch_bf16<64, true>(p.row_waves, grid, a, st);
      else launch_bf16<64, false>(p.row_waves, grid, a, st);
    }
  } else {
    if (d.head_dim == 128) launch_f32<128>(paged, grid, a, st);
    else launch_f32<64>(paged, grid, a, st);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.splits <= 1) return e;
  const int per_block = (p.rows_pb * d.head_dim / 4 + 255) / 256;
  const dim3 mgrid(per_block, d.num_kv_heads * p.row_blocks, d.batch);
  const bool bf16 = d.dtype == SIMSD_BF16;
  if (d.head_dim == 128) {
    if (bf16) hipLaunchKernelGGL((merge_kernel<128, uint16_t>), mgrid, dim3(256), 0, st, a);
    else hipLaunchKernelGGL((merge_kernel<128, float>), mgrid, dim3(256), 0, st, a);
  } else {
    if (bf16) hipLaunchKernelGGL((merge_kernel<64, uint16_t>), mgrid, dim3(256), 0, st, a);
    else hipLaunchKernelGGL((merge_kernel<64, float>), mgrid, dim3(256), 0, st, a);
  }
  return hipGetLastError();
}

}  // namespace simsd
