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
// sequence), or, for large ragged batches, one work-group per resident slot
// taking an equal range of all tiles (the stream decomposition).  The G query
// heads of a KV head and all B+L new slots are packed into the rows of one
// row block (GQA packing), so each K/V byte of the prefix is read from HBM
// once per KV head.  When a pair's keys are split over several work-groups,
// each writes a partial output with its running max and sum (bf16: the output
// normalised by its own sum, in bf16; fp32: unnormalised, in fp32), and a
// second kernel merges them; there is no device-wide fence or counter in the
// streaming kernel.
//
// bf16 path: K and V tiles of 64 keys stream into a ring of LDS tile slots
// with direct global->LDS loads issued up to three tiles ahead, so no
// registers hold data in flight; rows are XOR-swizzled in 16-byte chunks so
// that the reads below are free of bank conflicts.  Scores are computed
// transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16, so lane l owns query
// row l % 32 of its wave's 32-row block and a row's softmax state stays in two
// lanes (l, l ^ 32).  O^T = V^T P^T takes P straight from the score registers
// as the B operand; the V^T operand comes from LDS transpose reads
// (ds_read_b64_tr_b16), so no register shuffles are needed.  Row maxima are
// kept in log2 units and rescaled only when they grow by more than 2^8.
#include <algorithm>
#include <type_traits>

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

// Label of new slot `slot` given its block-slot step (ignored for reference
// slots).
__device__ inline SlotLabel slot_label(int slot, int step, int gamma, int B) {
  if (slot < B) {
    if (step < 0) return {-1, -1};
    return {0, step > gamma ? gamma + 1 : step};
  }
  const int r = slot - B;
  if (r >= gamma) return {-1, -1};
  return {1, r + 1};
}

// Whether a non-padded row with label li may attend to new slot lj.
__device__ inline bool slot_visible(SlotLabel li, SlotLabel lj) {
  if (lj.sec < 0) return false;
  if (lj.sec == 0 && lj.tau == 0) return true;
  if (li.sec == 1) return lj.sec == 1 ? lj.tau <= li.tau : lj.tau > li.tau;
  return lj.sec == 1 ? lj.tau < li.tau : lj.tau >= li.tau;
}

// Visibility words of the new slots, one 64-bit word per row (bit j: the row
// may attend to slot j; zero for padding rows), written to vis[0, n_new).
// Lane j holds slot j's label; row i's word is one ballot against the label
// of lane i.  `step` is lane j's block-slot step (any value for j >= B).
template <int NW>
__device__ inline void build_visibility(uint64_t* vis, int step, int gamma, int B, int n_new,
                                        int wave, int lane) {
  const SlotLabel lj = slot_label(lane, step, gamma, B);
  for (int i = wave; i < n_new; i += NW) {
    const SlotLabel li = {__builtin_amdgcn_readlane(lj.sec, i), __builtin_amdgcn_readlane(lj.tau, i)};
    const bool v = lane < n_new && li.sec >= 0 && slot_visible(li, lj);
    const uint64_t word = __ballot(v);
    if (lane == 0) vis[i] = word;
  }
}

// One contiguous key range of one (sequence, KV head, row block) pair that a
// work-group attends over: prefix keys [kbeg, kend), plus the new-slot tile
// when has_new.  A range that covers the whole pair (final) writes the
// normalised output; any other writes a partial (output, max, sum) to `part`.
struct Work {
  int split, kvh, rb, b, plen, nsplit, kbeg, kend, gamma;
  bool has_new, final;
  float* part;
};

__device__ inline float* partial_base(const AttnArgs& a, const Work& w, int D);

// Chunked decomposition: work-group (split, KV head x row block, sequence).
__device__ inline bool setup_work(const AttnArgs& a, Work& w, int D) {
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
  w.has_new = w.split == 0;
  w.final = w.nsplit == 1;
  w.part = w.final ? nullptr : partial_base(a, w, D);
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
// Rotary embedding (RoPE copy, Sec. 3.1-3.2).  Pair i of a head turns by
// pos * 2^(i * step) radians; the angle is formed in revolutions so that the
// hardware sine and cosine (period 1) apply after dropping whole turns.
constexpr float kInv2Pi = 0.15915494309189535f;
__device__ inline void rope_cs(int pos, int i, float step, float& c, float& s) {
  const float rev = static_cast<float>(pos) * (__builtin_amdgcn_exp2f(static_cast<float>(i) * step) * kInv2Pi);
  const float f = __builtin_amdgcn_fractf(rev);
  s = __builtin_amdgcn_sinf(f);
  c = __builtin_amdgcn_cosf(f);
}

// Positions of the new slots: block slot k at plen + k; reference slot r
// (draft r + 1) at its verification slot's index; padding reference slots at
// plen.  One wave; lane j holds block slot j's step.
__device__ inline void build_positions(int* s_pos, int step, int gamma, int B, int L, int plen,
                                       int lane) {
  if (lane < L) s_pos[B + lane] = plen;
  if (lane < B) {
    s_pos[lane] = plen + lane;
    if (step >= 1 && step <= gamma) s_pos[B + step - 1] = plen + lane;
  }
}

__device__ inline uint32_t pack2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Combine a value across lanes l and l ^ 32 (the two halves of an MFMA
// column) with one VALU lane swap instead of an LDS permute.  Both halves
// get the same bits (low half's value first).
__device__ inline float xhalf_max(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float xhalf_sum(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
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

constexpr int kMaxChunkPages = 2048;           // page ids of one key range staged in LDS

// Direct global -> LDS copy of 16 bytes per lane (global_load_lds_dwordx4):
// lane i's bytes land at LDS byte lds + 16 * i, so one instruction moves 1 KB.
// It counts in vmcnt like any vector load but the compiler does not track it:
// readers wait with wait_vm and then pass a barrier.  M0 (the LDS base) is a
// reserved register that the compiler does not allocate to values, so setting
// it here disturbs nothing.  dma16s takes a wave-uniform 64-bit base and a
// 32-bit per-lane offset (no per-lane address arithmetic).
__device__ inline void dma16(const void* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off"
               :: "v"(src), "s"(__builtin_amdgcn_readfirstlane(lds)) : "memory");
}
__device__ inline void dma16s(const void* base, uint32_t voff, uint32_t lds) {
  // readfirstlane works on (signed) int: each half goes through uint32_t
  // before widening so that the low half is not sign-extended.
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  const uint32_t hi = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b >> 32)));
  const uint32_t lo = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(b & 0xffffffffu)));
  const uint64_t bu = (static_cast<uint64_t>(hi) << 32) | lo;
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(bu), "s"(__builtin_amdgcn_readfirstlane(lds)) : "memory");
}
template <int N>
__device__ inline void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}
// This wave's LDS accesses complete, then a work-group barrier.  Unlike
// __syncthreads it does not wait for vector memory, so tiles still loading
// stay in flight.
__device__ inline void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Streams 64-key K/V tiles of one work-group's chunk into a ring of LDS tile
// slots with direct loads.  One instruction covers RPI key rows of one
// tensor; lane i writes chunk position i % CPR of row i / CPR of its block
// and so fetches logical chunk (i % CPR) ^ swz(row).  The tiles are split
// between the waves by instruction.  Full tiles (and the new-slot tile) use a
// wave-uniform base plus a fixed lane offset; rows past the prefix (the tail
// tile) or past the new slots read the last valid row instead: their scores
// are masked and their values are finite, so they add exact zeros.
template <int D, int NW, bool PAGED>
struct KVRing {
  static constexpr int ROWB = TileGeom<D>::ROWB, TILEB = TileGeom<D>::TILEB;
  static constexpr int CPR = D / 8;            // 16-byte chunks per key row
  static constexpr int RPI = 1024 / ROWB;      // key rows per instruction
  static constexpr int IPT = kTile / RPI;      // instructions per tensor per tile
  static constexpr int PERW = 2 * IPT / NW;    // instructions per wave per tile
  static_assert(PERW >= 1 && (2 * IPT) % NW == 0, "tile instructions split evenly over the waves");

  const char* kc;         // caches, offset to this KV head
  const char* vc;
  const char* kn;         // new slots, offset to (sequence, KV head, slot 0)
  const char* vn;
  int64_t seqoff;         // contiguous: this sequence's cache offset (bytes)
  int64_t tokb, pageb;    // bytes per token, per page
  int64_t newrow;         // bytes per new slot
  uint32_t voff[PERW];    // fast path: lane offset of instruction i (bytes)
  int row[PERW], chunk[PERW];
  int wave, P, lgP, pg_first, n_new;
  bool lds_pages;         // page ids of this chunk are staged in s_pg (P divides 64)
  bool fast;              // full tiles take the uniform-base path
  const int32_t* bt;      // this sequence's block table row

  __device__ __attribute__((always_inline)) void init(const AttnArgs& a, const Work& w, int wave_, int lane, SIMSD_LDS int* s_pg) {
    wave = wave_;
    const int64_t hoff = static_cast<int64_t>(w.kvh) * a.cs_head * 2;
    kc = static_cast<const char*>(a.k_cache) + hoff;
    vc = static_cast<const char*>(a.v_cache) + hoff;
    newrow = static_cast<int64_t>(a.hkv) * D * 2;
    const int64_t newoff = (static_cast<int64_t>(w.b) * a.n_new * a.hkv + w.kvh) * D * 2;
    kn = static_cast<const char*>(a.k_new) + newoff;
    vn = static_cast<const char*>(a.v_new) + newoff;
    tokb = a.cs_tok * 2;
    n_new = a.n_new;
    // Lane offsets of a tile must fit 32 bits: 64 rows of tokb bytes.
    fast = tokb < (int64_t{1} << 25);
    if (PAGED) {
      P = a.page_size;
      pageb = a.cs_seq * 2;
      bt = a.block_table + static_cast<int64_t>(w.b) * a.max_pages;
      pg_first = w.kbeg / P;
      const int npg = w.kend > w.kbeg ? (w.kend - 1) / P - pg_first + 1 : 0;
      lds_pages = (kTile % P == 0) && npg <= kMaxChunkPages;
      lgP = __builtin_ctz(P);                  // P is a power of two when it divides 64
      if (lds_pages)
        for (int j = wave * 64 + lane; j < npg; j += NW * 64) s_pg[j] = bt[pg_first + j];
      // One page per instruction: the instruction's RPI rows share a page.
      fast = fast && lds_pages && P % RPI == 0;
    } else {
      seqoff = static_cast<int64_t>(w.b) * a.cs_seq * 2;
    }
#pragma unroll
    for (int i = 0; i < PERW; ++i) {
      const int g = wave * PERW + i;
      row[i] = (g % IPT) * RPI + lane / CPR;
      chunk[i] = (lane % CPR) ^ swz<D>(row[i]);
      const int r = PAGED ? (P > 0 ? row[i] % P : 0) : row[i];
      voff[i] = static_cast<uint32_t>(static_cast<int64_t>(r) * tokb + chunk[i] * 16);
    }
  }

  // Byte offset of (key, element 0) from this head's cache base (general path).
  __device__ __attribute__((always_inline)) int64_t key_offset(int key, const SIMSD_LDS int* s_pg) const {
    if (!PAGED) return seqoff + static_cast<int64_t>(key) * tokb;
    // (s_pg is typed as LDS so that the compiler cannot fold the two reads
    // into one load through a generic pointer.)
    const int64_t page = lds_pages ? s_pg[key / P - pg_first] : bt[key / P];
    return page * pageb + static_cast<int64_t>(key % P) * tokb;
  }

  // Issue this wave's share of the tile starting at prefix key k0 (or of the
  // new-slot tile) into the ring slot at LDS byte address `slot`.
  __device__ __attribute__((always_inline)) void issue(uint32_t slot, int k0, bool is_new, int kend, const SIMSD_LDS int* s_pg) const {
    if (is_new) {
#pragma unroll
      for (int i = 0; i < PERW; ++i) {
        const int g = wave * PERW + i;
        const uint32_t off = static_cast<uint32_t>(min(row[i], n_new - 1) * newrow) + chunk[i] * 16;
        dma16s(g < IPT ? kn : vn, off, slot + (g / IPT) * TILEB + (g % IPT) * 1024);
      }
    } else if (k0 + kTile <= kend && fast) {
      // Paged: lane j holds page j of the tile (one LDS read); instruction i's
      // rows lie in one page (P is a multiple of RPI and k0 of P) and its lane
      // offsets hold the row within that page.
      int pgl = 0;
      if (PAGED) {
        const int j = min(static_cast<int>(threadIdx.x & 63), (kTile >> lgP) - 1);
        pgl = s_pg[((k0 - pg_first * P) >> lgP) + j];   // pg_first * P == kbeg
      }
#pragma unroll
      for (int i = 0; i < PERW; ++i) {
        const int g = wave * PERW + i;
        int64_t base;
        if (PAGED) base = static_cast<int64_t>(__builtin_amdgcn_readlane(pgl, ((g % IPT) * RPI) >> lgP)) * pageb;
        else base = seqoff + static_cast<int64_t>(k0) * tokb;
        dma16s((g < IPT ? kc : vc) + base, voff[i], slot + (g / IPT) * TILEB + (g % IPT) * 1024);
      }
    } else {
#pragma unroll
      for (int i = 0; i < PERW; ++i) {
        const int g = wave * PERW + i;
        const int key = min(k0 + row[i], kend - 1);
        const int64_t off = key_offset(key, s_pg) + chunk[i] * 16;
        dma16((g < IPT ? kc : vc) + off, slot + (g / IPT) * TILEB + (g % IPT) * 1024);
      }
    }
  }
};

// RW row waves of 32 rows each; KW = 2 pairs every row wave with a second wave
// that takes the other 32-key half of each tile (the stream decomposition and
// row blocks of up to 64 rows, where the extra waves double the work in
// flight); the two halves merge at the end.
// The ring holds NBUF tiles: tile it + NBUF - 1 loads while tile it is read.
// 8-wave groups have a CU to themselves (their registers allow no second
// group) and keep three tiles in flight; 4-wave groups keep a two-tile ring
// (measured faster than a deeper one: 3 or 4 tiles cost 13-17 % on the
// SDAR-8B layer with four whole-tile row waves, 10-35 % with two groups per
// CU).
template <int D, int RW, int KW, bool PAGED, bool ROPE>
__device__ __attribute__((always_inline)) void attend_segment(const AttnArgs& a, const Work& w) {
  constexpr int NW = RW * KW;
  constexpr int NBUF = NW >= 8 ? 4 : 2;
  constexpr int NB = D / 32;                   // 32-dim output blocks
  constexpr int KS = D / 16;                   // k-steps of QK^T
  constexpr int ROWB = TileGeom<D>::ROWB;
  constexpr int TILEB = TileGeom<D>::TILEB;
  using Ring = KVRing<D, NW, PAGED>;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[NBUF][2][TILEB];   // [slot][K, V]
  __shared__ uint64_t vis[kMaxNew];
  __shared__ int s_pos[kMaxNew];               // rotary positions of the new slots
  __shared__ int s_pg_arr[PAGED ? kMaxChunkPages : 1];
  SIMSD_LDS int* s_pg = (SIMSD_LDS int*)(&s_pg_arr[0]);

  __syncthreads();                             // the work-group's previous range is done with the LDS
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform
  const int n = lane & 31, h = lane >> 5;
  const int rw = wave % RW, kw = wave / RW;    // row wave, key half

  // This lane's block-slot step (slot = lane), for the visibility words.
  const int32_t* step_row = a.step_map + static_cast<int64_t>(w.b) * a.B;
  const int lane_step = step_row[min(lane, a.B - 1)];

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
  Ring kv;
  kv.init(a, w, wave, lane, s_pg);
  // Every load the compiler knows of (Q, the step map, page ids) completes
  // before the tile loads start: the compiler cannot see those, and a wait
  // of its own after them would wait for the whole ring.
  __builtin_amdgcn_s_waitcnt(0);
  if (PAGED) __syncthreads();                  // staged page ids

  const int ntp = w.kend > w.kbeg ? (w.kend - w.kbeg + kTile - 1) / kTile : 0;
  const int nt = ntp + (w.has_new ? 1 : 0);
  auto tile_k0 = [&](int it) { return w.kbeg + it * kTile; };
  const uint32_t ring0 = static_cast<uint32_t>(reinterpret_cast<uintptr_t>(
      (SIMSD_LDS void*)(&smem[0][0][0])));      // LDS byte address of slot 0
  constexpr uint32_t kSlotBytes = 2 * TILEB;
  // Every slot is free at the start: the first NBUF tiles load at once.
#pragma unroll
  for (int j = 0; j < NBUF; ++j)
    if (j < nt) kv.issue(ring0 + j * kSlotBytes, tile_k0(j), j == ntp, w.kend, s_pg);

  build_visibility<NW>(vis, lane_step, w.gamma, a.B, a.n_new, wave, lane);
  if (ROPE && wave == 0) build_positions(s_pos, lane_step, w.gamma, a.B, a.L, w.plen, lane);
  __syncthreads();                             // visibility words, positions
  const uint64_t myvis = row_in ? vis[t] : 0ull;
  if constexpr (ROPE) {
    // This lane's query dims 16*ks + 8*h + e (ks < KS/2) pair with the same
    // offsets in ks + KS/2; both halves sit in this lane.
    const int pos = s_pos[t];
#pragma unroll
    for (int ks = 0; ks < KS / 2; ++ks) {
      u32x4 lo = __builtin_bit_cast(u32x4, qop[ks]), hi = __builtin_bit_cast(u32x4, qop[ks + KS / 2]);
#pragma unroll
      for (int p = 0; p < 4; ++p) {
        float x1[2], x2[2], y1[2], y2[2];
        x1[0] = __uint_as_float(lo[p] << 16);
        x1[1] = __uint_as_float(lo[p] & 0xffff0000u);
        x2[0] = __uint_as_float(hi[p] << 16);
        x2[1] = __uint_as_float(hi[p] & 0xffff0000u);
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          float c, sn;
          rope_cs(pos, 16 * ks + 8 * h + 2 * p + e, a.rope_step, c, sn);
          y1[e] = x1[e] * c - x2[e] * sn;
          y2[e] = x2[e] * c + x1[e] * sn;
        }
        lo[p] = pack2(y1[0], y1[1]);
        hi[p] = pack2(y2[0], y2[1]);
      }
      qop[ks] = __builtin_bit_cast(bf16x8, lo);
      qop[ks + KS / 2] = __builtin_bit_cast(bf16x8, hi);
    }
  }

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

  // One tile: wait for it, free the slot of the previous tile for the next
  // load, then its key blocks.  `masked` tiles (the prefix tail and the
  // new-slot tile) take the mask code; full prefix tiles take a copy without
  // it.  `sl` is the tile's ring slot.
  auto tile = [&](auto masked, int it, int sl) __attribute__((always_inline)) {
    const bool is_new = it == ntp;
    const int k0 = tile_k0(it);
    // This wave's share of tile `it` has landed once at most the loads of the
    // younger tiles remain (vector memory completes in issue order).  Tiles
    // issued so far: the first NBUF, then one per earlier iteration.
    const int younger = min(nt - 1, max(NBUF - 1, it + NBUF - 2)) - it;
    if (NBUF >= 4 && younger >= 3) wait_vm<3 * Ring::PERW>();
    else if (NBUF >= 3 && younger >= 2) wait_vm<2 * Ring::PERW>();
    else if (younger >= 1) wait_vm<Ring::PERW>();
    else wait_vm<0>();
    lds_barrier();                             // all of tile `it` is in; slot of tile it-1 is free
    if (it >= 1 && it + NBUF - 1 < nt) {
      const int nx = it + NBUF - 1;
      kv.issue(ring0 + ((sl + NBUF - 1) % NBUF) * kSlotBytes, tile_k0(nx), nx == ntp, w.kend, s_pg);
    }
    // LDS-typed pointers (no generic-pointer arithmetic on the ring).
    const SIMSD_LDS uint8_t* sk = reinterpret_cast<const SIMSD_LDS uint8_t*>(ring0) + sl * kSlotBytes;
    const SIMSD_LDS uint8_t* sv = sk + TILEB;
    if (ROPE && decltype(masked)::value && is_new) {
      // Rotate the new keys in place: item (row r, chunk pair L) holds dims
      // 8L..8L+7 and their partners 8L + D/2.. (16-byte chunks L and L + CH/2,
      // swizzled).  Rows past the new slots hold copies of the last one.
      constexpr int CH = D / 8;
      SIMSD_LDS uint8_t* skw = const_cast<SIMSD_LDS uint8_t*>(sk);
      for (int item = tid; item < kTile * (CH / 2); item += NW * 64) {
        const int r = item / (CH / 2), L = item % (CH / 2);
        const int pos = s_pos[min(r, a.n_new - 1)];
        SIMSD_LDS u32x4* c1 = reinterpret_cast<SIMSD_LDS u32x4*>(skw + r * ROWB + 16 * (L ^ swz<D>(r)));
        SIMSD_LDS u32x4* c2 = reinterpret_cast<SIMSD_LDS u32x4*>(skw + r * ROWB + 16 * ((L + CH / 2) ^ swz<D>(r)));
        u32x4 lo = *c1, hi = *c2;
#pragma unroll
        for (int p = 0; p < 4; ++p) {
          float y1[2], y2[2];
#pragma unroll
          for (int e = 0; e < 2; ++e) {
            const float x1 = __uint_as_float(e ? (lo[p] & 0xffff0000u) : (lo[p] << 16));
            const float x2 = __uint_as_float(e ? (hi[p] & 0xffff0000u) : (hi[p] << 16));
            float c, sn;
            rope_cs(pos, 8 * L + 2 * p + e, a.rope_step, c, sn);
            y1[e] = x1 * c - x2 * sn;
            y2[e] = x2 * c + x1 * sn;
          }
          lo[p] = pack2(y1[0], y1[1]);
          hi[p] = pack2(y2[0], y2[1]);
        }
        *c1 = lo;
        *c2 = hi;
      }
      __syncthreads();
    }

    // The wave's key blocks of this tile, one at a time: both 32-key blocks
    // when KW == 1, block kw when KW == 2.  (Taking both blocks' scores at
    // once measured no faster and needs 16 more registers.)
#pragma unroll
    for (int kb1 = 0; kb1 < 2 / KW; ++kb1) {
    constexpr int NKB = 1;
    f32x16 s[NKB];
#pragma unroll
    for (int q = 0; q < NKB; ++q)
#pragma unroll
      for (int j = 0; j < 16; ++j) s[q][j] = 0.f;
    // S^T = K Q^T.  Register j of s[q] holds key 32*kb + 8*(j/4) + 4*h + j%4
    // of this lane's row, kb = the block of s[q].
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int q = 0; q < NKB; ++q) {
        const int kb = KW == 1 ? kb1 : kw;
        const bf16x8 ka = *reinterpret_cast<const SIMSD_LDS bf16x8*>(sk + 32 * kb * ROWB + koff[ks]);
        s[q] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ka, qop[ks], s[q], 0, 0, 0);
      }
    if constexpr (decltype(masked)::value) {
#pragma unroll
      for (int q = 0; q < NKB; ++q) {
        const int kb = KW == 1 ? kb1 : kw;
        if (is_new) {
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int key = 32 * kb + 8 * (j >> 2) + 4 * h + (j & 3);
            if (!((myvis >> key) & 1ull)) s[q][j] = kNegInf;
          }
        } else {
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int key = k0 + 32 * kb + 8 * (j >> 2) + 4 * h + (j & 3);
            if (key >= w.kend) s[q][j] = kNegInf;
          }
        }
      }
    }

    float mx = kNegInf;
#pragma unroll
    for (int q = 0; q < NKB; ++q)
#pragma unroll
      for (int j = 0; j < 16; ++j) mx = fmaxf(mx, s[q][j]);
    mx = xhalf_max(mx);
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
    for (int q = 0; q < NKB; ++q)
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const float p = __builtin_amdgcn_exp2f(fmaf(s[q][j], sl2, -moff));
        s[q][j] = p;
        l_run += p;
      }

    // O^T += V^T P^T, two 16-key chunks per block.  Chunk hf of block kb
    // covers keys 32*kb + 16*hf + kappa(h, i), kappa(h, i) = 8*(i/4) + 4*h + i%4.
#pragma unroll
    for (int q = 0; q < NKB; ++q) {
      const int kb = KW == 1 ? kb1 : kw;
#pragma unroll
      for (int hf = 0; hf < 2; ++hf) {
        u32x4 pw;
#pragma unroll
        for (int p = 0; p < 4; ++p) pw[p] = pack2(s[q][8 * hf + 2 * p], s[q][8 * hf + 2 * p + 1]);
        const bf16x8 pb = __builtin_bit_cast(bf16x8, pw);
        const SIMSD_LDS uint8_t* vblk = sv + (32 * kb + 16 * hf) * ROWB;
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
    }
  };

  // Full prefix tiles, unrolled by NBUF so that ring slots are compile-time
  // offsets; then the masked tiles (at most the prefix tail and the new slots).
  const int nfull = (w.kend - w.kbeg) / kTile;
  for (int it0 = 0; it0 < nfull; it0 += NBUF) {
#pragma unroll
    for (int u = 0; u < NBUF; ++u) {
      if (it0 + u >= nfull) break;
      tile(std::false_type{}, it0 + u, u);
    }
  }
  for (int it = nfull; it < nt; ++it) tile(std::true_type{}, it, it % NBUF);
  if constexpr (KW == 2) {
    __syncthreads();                           // the ring is free (no load is pending)
    // Merge the two key halves of each row through LDS (the tiles are free).
    constexpr int SLOT = NB * 16 + 2;
    SIMSD_LDS float* xs = reinterpret_cast<SIMSD_LDS float*>(ring0) + (rw * 64 + lane) * SLOT;
    if (kw == 1) {
#pragma unroll
      for (int c = 0; c < NB; ++c)
#pragma unroll
        for (int j = 0; j < 16; ++j) xs[c * 16 + j] = o[c][j];
      xs[NB * 16] = m_run;
      xs[NB * 16 + 1] = l_run;
    }
    __syncthreads();
    if (kw == 0) {
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
  }
  const float l_tot = xhalf_sum(l_run);
  // Register j of o[c] holds dim 32*c + 8*(j/4) + 4*h + j%4 of this row.
  if (row_in && (KW == 1 || kw == 0)) {
    if (w.final) {
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
    } else {
      // bf16 partial: this range's output normalised by its own sum (so in
      // the range of V), rounded to bf16; the max and the sum stay fp32.
      float* part = w.part;
      uint16_t* prow = reinterpret_cast<uint16_t*>(part) + rowl * D;
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
#pragma unroll
      for (int c = 0; c < NB; ++c)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const u32x2 v = {pack2(o[c][4 * q] * inv, o[c][4 * q + 1] * inv),
                           pack2(o[c][4 * q + 2] * inv, o[c][4 * q + 3] * inv)};
          *reinterpret_cast<u32x2*>(prow + 32 * c + 8 * q + 4 * h) = v;
        }
      if (h == 0) {
        part[a.rows_pb * D + rowl] = m_run;
        part[a.rows_pb * D + a.rows_pb + rowl] = l_tot;
      }
    }
  }
}

// Chunked decomposition: one work-group per (prefix chunk, KV head x row
// block, sequence).
template <int D, int RW, int KW, bool PAGED, bool ROPE>
__global__ void __launch_bounds__(RW * KW * 64, 2) attn_bf16_kernel(AttnArgs a) {
  Work w;
  if (!setup_work(a, w, D)) return;
  attend_segment<D, RW, KW, PAGED, ROPE>(a, w);
}

// Stream decomposition, for large and ragged batches.  The tiles of all
// pairs form one sequence: pair q = kvh * row_blocks + rb of sequence b owns
// tp_b consecutive tiles (its prefix tiles, then the new-slot tile) starting
// at seq0[b] + q * tp_b.  Work-group g of G takes tiles [g*T/G, (g+1)*T/G),
// so every group gets the same number of tiles however ragged the prefixes
// are (G = min(grid, T), so no range is empty); it attends over each pair's part of its range in turn.  A part that
// covers a whole pair writes the output; the others write partials to the
// group's two slots (0: the part at the start of its range, 1: the part at
// its end), which the merge kernel locates from the same arithmetic.
// seq0[0..batch] (int64) in LDS, and (group 0) in the workspace for the merge.
__device__ inline void stream_offsets(const AttnArgs& a, int64_t* seq0) {
  const int tid = threadIdx.x;
  const int pps = a.hkv * a.row_blocks;
  if (tid < kMaxStreamBatch) {
    int64_t v = 0;
    if (tid < a.batch) {
      const int plen = min(max(a.prefix_lens[tid], 0), a.max_prefix);
      v = static_cast<int64_t>(pps) * ((plen + kTile - 1) / kTile + 1);
    }
    seq0[tid + 1] = v;
  }
  if (tid == 0) seq0[0] = 0;
  __syncthreads();
  for (int off = 1; off < kMaxStreamBatch; off <<= 1) {   // inclusive scan of seq0[1..]
    const int64_t v = (tid < kMaxStreamBatch && tid >= off) ? seq0[1 + tid - off] : 0;
    __syncthreads();
    if (tid < kMaxStreamBatch) seq0[1 + tid] += v;
    __syncthreads();
  }
}

template <int D, int RW, int KW, bool PAGED, bool ROPE>
__global__ void __launch_bounds__(RW * KW * 64, 2) attn_bf16_stream(AttnArgs a) {
  __shared__ int64_t seq0[kMaxStreamBatch + 1];
  stream_offsets(a, seq0);
  // Every lane computes the same values from LDS; readfirstlane makes that
  // uniformity visible to the compiler (scalar registers, scalar branches).
  auto uni = [](int64_t v) {
    const uint32_t h = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(v >> 32)));
    const uint32_t l = static_cast<uint32_t>(__builtin_amdgcn_readfirstlane(static_cast<int>(v & 0xffffffff)));
    return static_cast<int64_t>((static_cast<uint64_t>(h) << 32) | l);
  };
  const int pps = a.hkv * a.row_blocks;
  const int64_t T = uni(seq0[a.batch]);
  const int g = blockIdx.x;
  if (g == 0)
    for (int i = threadIdx.x; i <= a.batch; i += blockDim.x) a.stream_seq0[i] = seq0[i];
  // With fewer tiles than groups only the first T groups work, so that every
  // working group's range is non-empty (the merge reads a slot of each).
  const int G = static_cast<int>(min<int64_t>(gridDim.x, T));
  if (g >= G) return;
  const int64_t lo = static_cast<int64_t>(g) * T / G, hi = static_cast<int64_t>(g + 1) * T / G;
  for (int64_t x = lo; x < hi;) {
    int b = 0;                                 // the sequence holding tile x
    for (int step = kMaxStreamBatch; step > 0; step >>= 1)
      if (b + step < a.batch && uni(seq0[b + step]) <= x) b += step;
    const int64_t s_b = uni(seq0[b]);
    const int64_t tp = (uni(seq0[b + 1]) - s_b) / pps;
    const int64_t local = x - s_b;
    const int q = static_cast<int>(local / tp);
    const int t0 = static_cast<int>(local % tp);
    const int t1 = static_cast<int>(min(tp, t0 + (hi - x)));
    const int ntp = static_cast<int>(tp) - 1;
    Work w;
    w.b = b;
    w.kvh = q / a.row_blocks;
    w.rb = q % a.row_blocks;
    w.split = 0;
    w.nsplit = 0;
    w.plen = min(max(a.prefix_lens[b], 0), a.max_prefix);
    w.gamma = min(max(a.num_ref[b], 0), a.L);
    w.kbeg = min(t0, ntp) * kTile;
    w.kend = min(min(t1, ntp) * kTile, w.plen);
    w.has_new = t1 == tp;
    w.final = t0 == 0 && t1 == tp;
    w.part = a.part + (static_cast<int64_t>(g) * 2 + (x == lo ? 0 : 1)) *
                          static_cast<int64_t>(a.rows_pb) * (D + 2);
    attend_segment<D, RW, KW, PAGED, ROPE>(a, w);
    x += t1 - t0;
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
  __shared__ int s_pos[kMaxNew];

  Work w;
  if (!setup_work(a, w, D)) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int32_t* step_row = a.step_map + static_cast<int64_t>(w.b) * a.B;
  const int lane_step = step_row[min(lane, a.B - 1)];
  build_visibility<NT / 64>(vis, lane_step, w.gamma, a.B, a.n_new, wave, lane);
  if (a.rope) {
    if (wave == 0) build_positions(s_pos, lane_step, w.gamma, a.B, a.L, w.plen, lane);
    __syncthreads();
  }
  // Rotary embedding of element e of a new slot's row x (fp64 angles: this is
  // the exact path): dims e and e +- D/2 form the pair.
  auto rotated = [&](const float* x, int e, int slot) -> float {
    const float v = x[e];
    if (!a.rope) return v;
    const int i = e % (D / 2);
    const float partner = x[e < D / 2 ? e + D / 2 : e - D / 2];
    const double ang = static_cast<double>(s_pos[slot]) * pow(static_cast<double>(a.rope_theta), -2.0 * i / D);
    const double c = cos(ang), sn = sin(ang);
    return static_cast<float>(e < D / 2 ? v * c - partner * sn : v * c + partner * sn);
  };
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
      v = rotated(static_cast<const float*>(a.q) + ((static_cast<int64_t>(w.b) * a.n_new + t) * a.hq + hq) * D, d, t);
    }
    sq[idx] = v;
    so[idx] = 0.f;
  }

  const float sl2 = a.scale_log2;
  const int ntp = w.kend > w.kbeg ? (w.kend - w.kbeg + TK - 1) / TK : 0;
  const int ntn = w.has_new ? (a.n_new + TK - 1) / TK : 0;
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
          const int64_t off = ((static_cast<int64_t>(w.b) * a.n_new + slot) * a.hkv + w.kvh) * D;
          kv = rotated(static_cast<const float*>(a.k_new) + off, e, slot);
          vv = static_cast<const float*>(a.v_new)[off + e];
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

  if (w.final) {
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
  float* part = w.part;
  for (int idx = tid; idx < 32 * D; idx += NT) part[idx] = so[idx];
  if (tid < 32) {
    part[a.rows_pb * D + tid] = sm[tid];
    part[a.rows_pb * D + a.rows_pb + tid] = sl[tid];
  }
}

// ----------------------------------------------------------------------------
// Merge of split partials.  Grid: (thread blocks over the packed rows of a row
// block, KV head x row block, sequence); one thread per (row, DPT dims of the
// output): 16 bytes of each partial, 8 dims of a bf16 partial or 4 of an fp32
// one, or 4 bf16 dims where many splits make each thread's loads long.
// Sequences whose prefix fits one chunk were finished by the attention kernel
// and are skipped.
// ----------------------------------------------------------------------------
// Merge of the partials of each pair.  Chunked decomposition: the pair's
// nsplit chunk partials.  Stream decomposition: the partials of the groups
// g_first..g_last whose tile ranges meet the pair (slot 1 of g_first when the
// pair starts inside its range, slot 0 otherwise); a pair inside one group's
// range was written whole by that group.
// SB partials are loaded per round (indices clamped, so a round always loads
// SB); the launcher takes SB near the split count.
template <int D, typename OutT, bool STREAM, int SB, int DPT = 16 / static_cast<int>(sizeof(OutT))>
__global__ void __launch_bounds__(256) merge_kernel(AttnArgs a) {
  static_assert(DPT == 4 || (DPT == 8 && sizeof(OutT) == 2), "dims per thread");
  constexpr int TPR = D / DPT;                                // threads per row
  // A zero the compiler cannot see through: keeps the per-sequence reads
  // vector loads issued with the others instead of late scalar loads.
  int lane_zero;
  asm volatile("v_mov_b32 %0, 0" : "=v"(lane_zero));
  const int b = blockIdx.z;
  const int kvh = blockIdx.y / a.row_blocks, rb = blockIdx.y % a.row_blocks;
  const int idx = blockIdx.x * 256 + threadIdx.x;
  const int rowl = idx / TPR, d0 = (idx % TPR) * DPT;
  // Rows past the packed rows of this block have no partials.
  if (rowl >= a.rows_pb || rb * a.rows_pb + rowl >= a.rows) return;
  const int rl = rowl;
  const int m = rb * a.rows_pb + rl;
  const int t = m / a.group, hq = kvh * a.group + m % a.group;

  // First round of loads, none waiting on another.  Indices are clamped so
  // every load is in bounds; split blocks past this sequence's count (stale
  // workspace) are loaded but never used.
  const int nref = a.num_ref[b + lane_zero];
  const int step = a.step_map[static_cast<int64_t>(b) * a.B + min(t, a.B - 1)];
  const int64_t pstride = static_cast<int64_t>(a.rows_pb) * (D + 2);
  const int mo = a.rows_pb * D;
  int nsplit;
  const float* base = a.part;
  int g_first = 0, G = 1;
  int64_t start = 0, T = 1;
  if constexpr (STREAM) {
    const int64_t sb = a.stream_seq0[b + lane_zero], se = a.stream_seq0[b + 1 + lane_zero];
    T = a.stream_seq0[a.batch + lane_zero];
    G = static_cast<int>(min<int64_t>(a.stream_groups, T));   // the working groups
    const int64_t tp = (se - sb) / (a.hkv * a.row_blocks);
    start = sb + static_cast<int64_t>(kvh * a.row_blocks + rb) * tp;
    // owner(x) = the group g with g*T/G <= x < (g+1)*T/G
    g_first = static_cast<int>(((start + 1) * G - 1) / T);
    const int g_last = static_cast<int>(((start + tp) * G - 1) / T);
    nsplit = g_last - g_first + 1;
  } else {
    const int plen = min(max(a.prefix_lens[b + lane_zero], 0), a.max_prefix);
    nsplit = plen > 0 ? (plen + a.chunk - 1) / a.chunk : 1;
    base += ((static_cast<int64_t>(b) * a.hkv + kvh) * a.row_blocks + rb) * a.splits * pstride;
  }
  auto part_of = [&](int s) -> const float* {
    if constexpr (STREAM) {
      s = min(s, nsplit - 1);
      const int g = g_first + s;
      const int slot = (s == 0 && static_cast<int64_t>(g) * T / G < start) ? 1 : 0;
      return base + (static_cast<int64_t>(g) * 2 + slot) * pstride;
    } else {
      return base + min(s, a.splits - 1) * pstride;
    }
  };
  float mv[SB], lv[SB];
  float ov[SB][DPT];
  auto load_round = [&](int s0) {
#pragma unroll
    for (int s = 0; s < SB; ++s) {
      const float* ps = part_of(s0 + s);
      mv[s] = ps[mo + rl];
      lv[s] = ps[mo + a.rows_pb + rl];
      if constexpr (sizeof(OutT) == 2 && DPT == 8) {   // bf16 partials, normalised by their sum
        const u32x4 w4 = *reinterpret_cast<const u32x4*>(reinterpret_cast<const uint16_t*>(ps) + rl * D + d0);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          ov[s][2 * e] = __uint_as_float(w4[e] << 16);
          ov[s][2 * e + 1] = __uint_as_float(w4[e] & 0xffff0000u);
        }
      } else if constexpr (sizeof(OutT) == 2) {
        const u32x2 w2 = *reinterpret_cast<const u32x2*>(reinterpret_cast<const uint16_t*>(ps) + rl * D + d0);
#pragma unroll
        for (int e = 0; e < 2; ++e) {
          ov[s][2 * e] = __uint_as_float(w2[e] << 16);
          ov[s][2 * e + 1] = __uint_as_float(w2[e] & 0xffff0000u);
        }
      } else {
        const f32x4 f4 = *reinterpret_cast<const f32x4*>(ps + rl * D + d0);
#pragma unroll
        for (int e = 0; e < 4; ++e) ov[s][e] = f4[e];
      }
    }
  };
  if (!STREAM) load_round(0);                  // chunked: before the split count is known
  if (nsplit <= 1) return;
  if (STREAM) load_round(0);
  const int gamma = min(max(nref, 0), a.L);
  // A row is padding iff it sees no new slot (a non-padded row always sees itself).
  const bool valid = t < a.B ? step >= 0 : (t - a.B) < gamma;

  float mt = kNegInf, lsum = 0.f;
  float acc[DPT];
#pragma unroll
  for (int e = 0; e < DPT; ++e) acc[e] = 0.f;
  for (int s0 = 0; s0 < nsplit; s0 += SB) {
    if (s0 > 0) load_round(s0);
    float mb = kNegInf;
#pragma unroll
    for (int s = 0; s < SB; ++s)
      if (s0 + s < nsplit) mb = fmaxf(mb, mv[s]);
    const float mn = fmaxf(mt, mb);
    if (mn == kNegInf) continue;
    const float alpha = __builtin_amdgcn_exp2f(mt - mn);   // 0 while mt is -inf
    lsum *= alpha;
#pragma unroll
    for (int e = 0; e < DPT; ++e) acc[e] *= alpha;
#pragma unroll
    for (int s = 0; s < SB; ++s) {
      if (s0 + s < nsplit) {
        const float wt = __builtin_amdgcn_exp2f(mv[s] - mn);
        lsum += wt * lv[s];
        // bf16 partials hold O / l: their weight carries the sum.
        const float wo = sizeof(OutT) == 2 ? wt * lv[s] : wt;
#pragma unroll
        for (int e = 0; e < DPT; ++e) acc[e] += wo * ov[s][e];
      }
    }
    mt = mn;
  }
  const bool ok = valid && lsum > 0.f;
  const float inv = ok ? 1.f / lsum : 0.f;
  const int64_t orow = ((static_cast<int64_t>(b) * a.n_new + t) * a.hq + hq) * D + d0;
  if constexpr (sizeof(OutT) == 2 && DPT == 8) {
    const u32x4 pk = {pack2(acc[0] * inv, acc[1] * inv), pack2(acc[2] * inv, acc[3] * inv),
                      pack2(acc[4] * inv, acc[5] * inv), pack2(acc[6] * inv, acc[7] * inv)};
    *reinterpret_cast<u32x4*>(static_cast<uint16_t*>(a.out) + orow) = pk;
  } else if constexpr (sizeof(OutT) == 2) {
    const u32x2 pk = {pack2(acc[0] * inv, acc[1] * inv), pack2(acc[2] * inv, acc[3] * inv)};
    *reinterpret_cast<u32x2*>(static_cast<uint16_t*>(a.out) + orow) = pk;
  } else {
    *reinterpret_cast<f32x4*>(static_cast<float*>(a.out) + orow) =
        f32x4{acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv};
  }
  if (d0 == 0 && a.lse)
    a.lse[(static_cast<int64_t>(b) * a.hq + hq) * a.n_new + t] =
        ok ? (mt + __log2f(lsum)) * kLn2 : kNegInf;
}

template <int D, bool PAGED, bool ROPE>
void launch_bf16_variant(const AttnPlan& p, dim3 grid, const AttnArgs& a, hipStream_t st) {
  if (p.stream) {
    const dim3 sg(p.stream_groups);
    switch (p.row_waves) {
      case 2: hipLaunchKernelGGL((attn_bf16_stream<D, 2, 2, PAGED, ROPE>), sg, dim3(256), 0, st, a); break;
      default: hipLaunchKernelGGL((attn_bf16_stream<D, 4, 2, PAGED, ROPE>), sg, dim3(512), 0, st, a); break;
    }
    return;
  }
  switch (p.row_waves) {
    case 2: hipLaunchKernelGGL((attn_bf16_kernel<D, 2, 2, PAGED, ROPE>), grid, dim3(256), 0, st, a); break;
    case 4:
      // The rotary variant of four whole-tile row waves needs more registers
      // than two groups per CU allow; it spilled the tile loads' lane offsets,
      // and each reload's wait drained the ring (SDAR-8B layer with RoPE 70.5
      // against 45.3 us for the 8-wave half-tile groups).
      if constexpr (ROPE) hipLaunchKernelGGL((attn_bf16_kernel<D, 4, 2, PAGED, ROPE>), grid, dim3(512), 0, st, a);
      else hipLaunchKernelGGL((attn_bf16_kernel<D, 4, 1, PAGED, ROPE>), grid, dim3(256), 0, st, a);
      break;
    default: hipLaunchKernelGGL((attn_bf16_kernel<D, 8, 1, PAGED, ROPE>), grid, dim3(512), 0, st, a); break;
  }
}

// The rotary variants are separate instantiations: their extra registers stay
// out of the kernels that run without it.
template <int D, bool PAGED>
void launch_bf16(const AttnPlan& p, dim3 grid, const AttnArgs& a, hipStream_t st) {
  if (a.rope) launch_bf16_variant<D, PAGED, true>(p, grid, a, st);
  else launch_bf16_variant<D, PAGED, false>(p, grid, a, st);
}

// Chunked merge: loads per round near the split count; above 8 splits each
// thread takes 4 dims (twice the threads, half the registers per load round).
template <int D, typename OutT>
void launch_merge(int splits, dim3 grid, const AttnArgs& a, hipStream_t st) {
  if (splits <= 2) hipLaunchKernelGGL((merge_kernel<D, OutT, false, 2>), grid, dim3(256), 0, st, a);
  else if (splits <= 4) hipLaunchKernelGGL((merge_kernel<D, OutT, false, 4>), grid, dim3(256), 0, st, a);
  else if (splits <= 8) hipLaunchKernelGGL((merge_kernel<D, OutT, false, 8>), grid, dim3(256), 0, st, a);
  else hipLaunchKernelGGL((merge_kernel<D, OutT, false, 16, 4>), grid, dim3(256), 0, st, a);
}

// Dims per merge thread (see merge_kernel).
inline int merge_dims(const AttnPlan& p, bool bf16) {
  return bf16 && (p.stream || p.splits <= 8) ? 8 : 4;
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
      if (paged) launch_bf16<128, true>(p, grid, a, st);
      else launch_bf16<128, false>(p, grid, a, st);
    } else {
      if (paged) launch_bf16<64, true>(p, grid, a, st);
      else launch_bf16<64, false>(p, grid, a, st);
    }
  } else {
    if (d.head_dim == 128) launch_f32<128>(paged, grid, a, st);
    else launch_f32<64>(paged, grid, a, st);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || (p.splits <= 1 && !p.stream)) return e;
  // Threads for the packed rows only (the last row block may be partial), one
  // per merge_dims() dims of a row.
  const bool bf16 = d.dtype == SIMSD_BF16;
  const int per_block = (std::min(p.rows_pb, p.rows) * d.head_dim / merge_dims(p, bf16) + 255) / 256;
  const dim3 mgrid(per_block, d.num_kv_heads * p.row_blocks, d.batch);
  if (p.stream) {
    // A pair meets a few group ranges (two or three on the ragged batches);
    // more take further rounds.
    if (d.head_dim == 128) hipLaunchKernelGGL((merge_kernel<128, uint16_t, true, 4>), mgrid, dim3(256), 0, st, a);
    else hipLaunchKernelGGL((merge_kernel<64, uint16_t, true, 4>), mgrid, dim3(256), 0, st, a);
  } else if (d.head_dim == 128) {
    if (bf16) launch_merge<128, uint16_t>(p.splits, mgrid, a, st);
    else launch_merge<128, float>(p.splits, mgrid, a, st);
  } else {
    if (bf16) launch_merge<64, uint16_t>(p.splits, mgrid, a, st);
    else launch_merge<64, float>(p.splits, mgrid, a, st);
  }
  return hipGetLastError();
}

}  // namespace simsd
