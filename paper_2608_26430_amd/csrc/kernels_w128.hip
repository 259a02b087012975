// Fused forward / backward for frames whose diagonal block is 128 x 128
// (k = 64, e.g. every 4096-wide Llama projection with rho = 64), bf16
// activations.
//
// Layout.  A workgroup owns a tile of 8 tokens.  The coefficients of one side
// (z = P_in^T x forward, u = P_out^T g backward) live in LDS coefficient-major:
// row c holds the 8 tokens' bf16 values (16 bytes), so every sparse access of
// C's random support is one 16-byte LDS read covering the whole tile.  The
// analysis that fills these arrays runs the MFMA with its operands swapped, so
// that each lane ends up with four tokens of one coefficient and writes them
// with a single 8-byte store.  The per-wave pair tiles, which the synthesis
// reads as MFMA operands (8 consecutive coefficients of one token), are
// XOR-swizzled inside each 128-row block so that those reads hit distinct
// banks.  In a partial tile (fewer than 8 tokens left) the missing
// token columns repeat the last token: every result they produce equals that
// token's and is written to that token's row, so no store needs a lane mask;
// only the dC products mask them out.
//
// Frame products.  Only the upper half of the block B (synthesis) is held in
// registers (64 VGPRs per wave, staged once per workgroup through LDS): the
// lower half is the upper half applied to the input with its odd complex
// components negated, B[u + 64][c] = (-1)^(c/2) B[u][c], the row-wise radix-2
// symmetry of the DFT.  Analysis needs B^T; for these frames B^T = D B D with
// D = diag(+1, -1, +1, ...) (the realified DFT is symmetric up to the sign of
// its sine terms), so analysis negates odd inputs and odd outputs and reuses
// the same fragments.  All sign changes are XORs on the packed bf16 operand.
// One v_mfma_f32_16x16x32_bf16 column group is 16 (token, block) pairs: 8
// tokens times a pair of blocks.
//
// Sparse products.  After the shared coefficient array is complete, each wave
// streams over its own block pairs with a private 4 KB LDS tile.  The plan's
// entry streams are load-balanced and lane-interleaved (a lane owns whole rows
// of C for v = C z, whole columns for q = C^T u), every stream has at least one
// row, and the coefficient vector is laid out like the forward stream (slot
// (row r, lane l) is coefficient 64 r + l), so forward slots read their
// coefficients with coalesced loads that do not wait for the entries.  A
// chunk's LDS reads are all issued before its sums and its row writes, so one
// LDS latency is paid per chunk rather than per slot.  The sparse products
// multiply bf16 values by the coefficient rounded to bf16 with
// v_dot2_f32_bf16 against (c, 0) and (0, c), which takes each token straight
// from its packed pair, and accumulate in fp32.  The backward runs one
// stream per input pair twice: first for this tile's share of
// dC_e = sum_t u_t[a_e] z_t[b_e] (v_dot2_f32_bf16 over token pairs), then for
// q = C^T u; partial dC sums go to a workspace reduced in a fixed order by a
// second kernel.
//
// Memory-latency discipline.  The vector memory counter is in order and counts
// stores as well as loads, so waiting for a load also waits for every store
// issued before it, and a load that only some paths issue forces the compiler
// into full waits.  Hence: every prefetch is issued on every path (out-of-range
// pairs are clamped to a valid one and the result discarded), partial-sum
// stores of slots past a stream's end go to a scratch row instead of being
// skipped, the rare long-stream paths end with an explicit full wait, the
// output options are template parameters rather than branches, and the loads a
// pair needs are issued before the previous pair's stores.
#include <type_traits>

#include "ff_internal.h"

namespace ff {
namespace {

constexpr int kW = 128;   // block width
constexpr int kTT = 8;    // tokens per tile
constexpr int kMT = 8;    // 16-row output tiles per block
constexpr int kHT = kMT / 2;   // 16-row tiles of the upper half (held in registers)
constexpr int kKT = 4;    // 32-wide contraction steps per block
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
constexpr int kCh = 12;   // stream slots per lane held in registers at once


typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned short u16;
typedef short i16x4 __attribute__((ext_vector_type(4)));

// Global-memory views of generic pointers.  Pointers read from device arrays (the batched
// entry points) carry no address space, and loads through them would be emitted as flat
// loads, which the compiler must fence with full waits; every global access goes through
// these casts so that it is a global load or store.
#define FF_GLOBAL __attribute__((address_space(1)))
template <typename T>
__device__ __forceinline__ const FF_GLOBAL T* gld(const T* p) {
  return (const FF_GLOBAL T*)p;
}
template <typename T>
__device__ __forceinline__ FF_GLOBAL T* gst(T* p) {
  return (FF_GLOBAL T*)p;
}

__device__ __forceinline__ float lo_bf(unsigned w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf(unsigned w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ unsigned pack_bf2(float a, float b) {
  bf16x2 p = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(unsigned, p);
}

__device__ __forceinline__ u16 to_bf(float a) { return __builtin_bit_cast(u16, (__bf16)a); }

// s_waitcnt vmcnt(0), other counters untouched: ends a rare path with no vector memory
// operation of it still in flight.
__device__ __forceinline__ void vm_wait_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// Ordering point between phases that hand data through a wave's private LDS tile:
// LDS instructions of one wave execute in order, so only the compiler must not move
// accesses across it.
__device__ __forceinline__ void wave_lds_fence() { __asm__ volatile("" ::: "memory"); }

// A scheduling barrier: no instruction moves across it.  Placed after each group of
// prefetch loads, it keeps them where they are written (the scheduler would otherwise move
// them down next to their use, or hoist the arithmetic that consumes the previous prefetch
// above the work that was meant to hide its latency).
__device__ __forceinline__ void issue_point() { __builtin_amdgcn_sched_barrier(0); }

struct Frag {
  bf16x8 f[kHT][kKT];
};

// The 16 KB of upper-half synthesis fragments are fetched by the whole workgroup (NTH
// threads, 16 KB / NTH per thread, issued before anything else the kernel loads), staged
// through LDS and read back by every wave.  The fragment array is ordered [row tile][contraction
// step][lane], so the upper half is its first half.
template <int NTH>
constexpr int frag_per_thread() { return kHT * kKT * 64 / NTH; }
constexpr int kFragPerThread = frag_per_thread<kThreads>();

template <int NTH = kThreads>
__device__ __forceinline__ void frag_fetch(const void* fs16, u32x4 (&r)[frag_per_thread<NTH>()]) {
  const FF_GLOBAL u32x4* src = gld(reinterpret_cast<const u32x4*>(fs16));
#pragma unroll
  for (int j = 0; j < frag_per_thread<NTH>(); ++j) r[j] = src[threadIdx.x + j * NTH];
}

// `stage` must be free LDS of 16 KB; it may be reused after return.
template <int NTH = kThreads>
__device__ __forceinline__ void frag_stage(const u32x4 (&r)[frag_per_thread<NTH>()], u32x4* stage, int lane,
                                           Frag& F) {
#pragma unroll
  for (int j = 0; j < frag_per_thread<NTH>(); ++j) stage[threadIdx.x + j * NTH] = r[j];
  __syncthreads();
#pragma unroll
  for (int mt = 0; mt < kHT; ++mt)
#pragma unroll
    for (int ks = 0; ks < kKT; ++ks) F.f[mt][ks] = __builtin_bit_cast(bf16x8, stage[(mt * kKT + ks) * 64 + lane]);
  __syncthreads();
}

// Synthesis: acc[mt] = sum_ks B[mt][ks] * b[ks] for the 8 row tiles of the block; rows
// 64..127 use the upper-half fragments on the input with its odd complex components negated.
// A lane's 8 inputs of a contraction step are real indices 32 ks + 8 q + j: odd j is the high
// half of each word, odd complex index is words 1 and 3.
__device__ __forceinline__ void mfma_block(const Frag& F, const u32x4 (&b)[kKT], f32x4 (&acc)[kMT]) {
  const u32x4 m_bot = {0u, 0x80008000u, 0u, 0x80008000u};
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < kKT; ++ks) {
    const bf16x8 bt = __builtin_bit_cast(bf16x8, b[ks]);
    const bf16x8 bb = __builtin_bit_cast(bf16x8, b[ks] ^ m_bot);
#pragma unroll
    for (int mt = 0; mt < kHT; ++mt) {
      acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(F.f[mt][ks], bt, acc[mt], 0, 0, 0);
      acc[mt + kHT] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(F.f[mt][ks], bb, acc[mt + kHT], 0, 0, 0);
    }
  }
}

// Analysis with the operands swapped: D^T = X^T B^T, so lane (q, n) ends up holding
// coefficient 16 mt + n (mt < 4: upper half of the block, mt >= 4: lower half) of block
// (q >> 1) of the pair for tokens 4 (q & 1) .. 4 (q & 1) + 3.  Odd real inputs are negated
// (B^T = D B D); `km` zeroes the activation columns of tokens past the tile's end where they
// must not contribute.
__device__ __forceinline__ void mfma_block_t(const Frag& F, const u32x4 (&b)[kKT], f32x4 (&acc)[kMT], unsigned km) {
  const unsigned d = 0x80000000u;
  const u32x4 m_top = {d, d, d, d};
  const u32x4 m_bot = {d, d ^ 0x80008000u, d, d ^ 0x80008000u};
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < kKT; ++ks) {
    const u32x4 bk = b[ks] & km;
    const bf16x8 bt = __builtin_bit_cast(bf16x8, bk ^ m_top);
    const bf16x8 bb = __builtin_bit_cast(bf16x8, bk ^ m_bot);
#pragma unroll
    for (int mt = 0; mt < kHT; ++mt) {
      acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bt, F.f[mt][ks], acc[mt], 0, 0, 0);
      acc[mt + kHT] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bb, F.f[mt][ks], acc[mt + kHT], 0, 0, 0);
    }
  }
}

// Store the result of mfma_block_t into a coefficient-major LDS array of 16-byte rows (odd
// coefficients negated: sgn = 0x80008000 on lanes with odd n), one 8-byte write per row tile at
// `row` (this lane's byte offset in row tile 0) + 256 mt.
__device__ __forceinline__ void store_coef_t(unsigned char* lds, unsigned row, const f32x4 (&acc)[kMT],
                                             unsigned sgn) {
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt) {
    const unsigned w0 = pack_bf2(acc[mt][0], acc[mt][1]) ^ sgn, w1 = pack_bf2(acc[mt][2], acc[mt][3]) ^ sgn;
    *reinterpret_cast<u32x2*>(lds + row + 256 * mt) = u32x2{w0, w1};
  }
}

// Pair tile: 128 rows of 32 bytes, one per coefficient k of the block width, each holding the
// 8 tokens of both blocks.  Within 32 coefficients the rows are ordered by (bit 2, bits 3..4,
// bits 0..1) of k, so that one transposed read of the synthesis operand covers 512 contiguous
// bytes, and rows with bit 2 of k set hold block 1 in their first half.  Byte offset of this
// lane's 8 bytes of row tile 0 of mfma_block_t's result (lane: coefficient n of quarter q, whose
// 4 tokens are half q & 1 of block q >> 1), and the offset that row tile mt adds.
__device__ __forceinline__ unsigned tile_lane_off(int lane) {
  const int n = lane & 15, q = lane >> 4, b2 = (n >> 2) & 1;
  return 512 * b2 + 128 * (n >> 3) + 32 * (n & 3) + 8 * (q ^ (2 * b2));
}
__device__ __forceinline__ constexpr unsigned tile_mt_off(int mt) { return 1024 * (mt >> 1) + 256 * (mt & 1); }

// Store the result of mfma_block_t into the pair tile (odd coefficients negated as in
// store_coef_t); 32 lanes of one write cover 256 distinct bytes.
__device__ __forceinline__ void store_tile_t(unsigned char* tile, unsigned off, const f32x4 (&acc)[kMT],
                                             unsigned sgn) {
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt) {
    const unsigned w0 = pack_bf2(acc[mt][0], acc[mt][1]) ^ sgn, w1 = pack_bf2(acc[mt][2], acc[mt][3]) ^ sgn;
    *reinterpret_cast<u32x2*>(tile + off + tile_mt_off(mt)) = u32x2{w0, w1};
  }
}

// Activation fragments of one column group: lane (token t, block bs of the pair, quarter q)
// reads 8 consecutive inputs per contraction step from a row-major token matrix.  Token
// columns past the tile's end read its last token.
__device__ __forceinline__ void load_act(const u16* rows, long ld, int nt, int blk0, int lane, u32x4 (&b)[kKT]) {
  const int n = lane & 15, t = min(n & 7, nt - 1), bs = n >> 3, q = lane >> 4;
  const FF_GLOBAL u32x4* p = gld(reinterpret_cast<const u32x4*>(rows + (long)t * ld + (blk0 + bs) * kW + 8 * q));
#pragma unroll
  for (int ks = 0; ks < kKT; ++ks) b[ks] = p[4 * ks];
}

// The synthesis operand from the pair tile by transposed LDS reads (ds_read_b64_tr_b16): in each
// 16-lane group the lanes' 8-byte chunks form 4 rows of 16 bf16 values and lane i receives
// value i of each row.  Lane (column n = 8 bs + t, quarter q) thus receives token t of block bs
// at 4 consecutive coefficients per read; read h of step ks covers coefficients
// 32 ks + 8 q + 4 h + (0..3), the 16 tile rows starting at row 32 ks + 16 h, whose halves are
// swapped when h = 1.
__device__ __forceinline__ void load_tile_act(const unsigned char* tile, int lane, u32x4 (&b)[kKT]) {
#pragma unroll
  for (int ks = 0; ks < kKT; ++ks) {
    u32x2 v[2];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      auto* p = (__attribute__((address_space(3))) i16x4*)(const_cast<unsigned char*>(tile) +
                                                           (32 * ks + 16 * h) * 32 + 8 * (lane ^ (2 * h)));
      v[h] = __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(p));
    }
    b[ks] = u32x4{v[0].x, v[0].y, v[1].x, v[1].y};
  }
}

// y[t][(blk0+bs)*128 + o] = acc (+ beta * y); the scale s is already in the coefficients.  Token
// columns past the tile's end hold the last token's values and write them to its row again.
// Without beta the result is first transposed through the wave's pair tile (free at this point),
// so that each store instruction writes four whole 256-byte token rows rather than sixteen 32-byte
// pieces: tile row n = 8 bs + t holds the row's 16-byte chunks c at position c ^ n, which keeps
// both the 8-byte writes of one row tile and the 16-byte reads of one token row on distinct banks.
// With beta the old values are added in fp32 before the only rounding, so that path stores
// directly.
template <bool BETA>
__device__ __forceinline__ void store_act(u16* rows, long ld, int nt, int blk0, int lane, const f32x4 (&acc)[kMT],
                                          float beta, unsigned char* tile) {
  if constexpr (!BETA) {
    const int n = lane & 15, q = lane >> 4;
    wave_lds_fence();
#pragma unroll
    for (int mt = 0; mt < kMT; ++mt) {
      const unsigned pos = (unsigned)((2 * mt + (q >> 1)) ^ n);
      *reinterpret_cast<u32x2*>(tile + n * 256 + pos * 16 + 8 * (q & 1)) =
          u32x2{pack_bf2(acc[mt][0], acc[mt][1]), pack_bf2(acc[mt][2], acc[mt][3])};
    }
    wave_lds_fence();
    u32x4 v[4];
    const int c = lane & 15;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 4 * i + (lane >> 4);
      v[i] = *reinterpret_cast<const u32x4*>(tile + r * 256 + (unsigned)(c ^ r) * 16);
    }
    wave_lds_fence();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int r = 4 * i + (lane >> 4), t = min(r & 7, nt - 1), bs = r >> 3;
      *gst(reinterpret_cast<u32x4*>(rows + (long)t * ld + (blk0 + bs) * kW + 8 * c)) = v[i];
    }
  } else {
    const int n = lane & 15, t = min(n & 7, nt - 1), bs = n >> 3, q = lane >> 4;
    FF_GLOBAL u32x2* p = gst(reinterpret_cast<u32x2*>(rows + (long)t * ld + (blk0 + bs) * kW + 4 * q));
    u32x2 old[kMT];
#pragma unroll
    for (int mt = 0; mt < kMT; ++mt) old[mt] = p[4 * mt];
#pragma unroll
    for (int mt = 0; mt < kMT; ++mt) {
      f32x4 r = acc[mt];
      r[0] += beta * lo_bf(old[mt].x);
      r[1] += beta * hi_bf(old[mt].x);
      r[2] += beta * lo_bf(old[mt].y);
      r[3] += beta * hi_bf(old[mt].y);
      p[4 * mt] = u32x2{pack_bf2(r[0], r[1]), pack_bf2(r[2], r[3])};
    }
  }
}

// Wave priority by progress (`steps` = this wave's share of the phase, `done` = steps finished):
// the waves with more left issue first, so the two workgroups that share a CU advance together
// instead of the older one finishing first and leaving the other to run alone.
__device__ __forceinline__ void prio_by_progress(int done, int steps) {
  const int left = steps - done;   // wave-uniform
  if (4 * left > 3 * steps) __builtin_amdgcn_s_setprio(3);
  else if (2 * left > steps) __builtin_amdgcn_s_setprio(2);
  else if (4 * left > steps) __builtin_amdgcn_s_setprio(1);
  else __builtin_amdgcn_s_setprio(0);
}

__device__ __forceinline__ void zero_tile(unsigned char* tile, int lane) {
  u32x4* tz = reinterpret_cast<u32x4*>(tile);
  wave_lds_fence();
#pragma unroll
  for (int i = 0; i < 4; ++i) tz[lane + 64 * i] = u32x4{0u, 0u, 0u, 0u};
  wave_lds_fence();
}

// The coefficient-array row named by a slot word's source field.  The array starts the
// kernels' dynamic LDS, which has no static LDS before it, so the field is the LDS address.
__device__ __forceinline__ u32x4 lds_src(unsigned e) {
  return *(const __attribute__((address_space(3))) u32x4*)(size_t)(e & kSlotSrcMask);
}

__device__ __forceinline__ u32x4 lds_at(const unsigned char* base, unsigned byte_off) {
  return *reinterpret_cast<const u32x4*>(base + byte_off);
}

__device__ __forceinline__ unsigned tile_off(unsigned e) { return e >> kSlotDstShift; }

// The scaled coefficient of a slot as the two multiplier words of v_dot2_f32_bf16, (s c, 0) and
// (0, s c).  Padding slots have zero coefficients and add nothing.
__device__ __forceinline__ void coef_words(float c, float scale, unsigned& ce, unsigned& co) {
  // one conversion with a constant zero low half (the compiler builds (0, x) from two words)
  asm("v_cvt_pk_bf16_f32 %0, 0, %1" : "=v"(co) : "v"(c * scale));
  ce = co >> 16;
}

__device__ __forceinline__ float dot2(unsigned a, unsigned b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, a), __builtin_bit_cast(bf16x2, b), c, false);
}

// a[t] += c z[t] for the 8 tokens of one source row.  At a round end (`end`, the same on every
// lane) every lane writes its current row to the tile position named by its slot word, and
// restarts it if the row ends with this round (a row that goes on is written again later).
__device__ __forceinline__ void accum_slot(unsigned e, unsigned ce, unsigned co, const u32x4 zv, bool end,
                                           unsigned char* tile, float (&a)[8]) {
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    // copy the element out first: bit-casting a vector element expression directly reads
    // element 0 with this compiler
    const unsigned w = zv[j];
    a[2 * j] = dot2(w, ce, a[2 * j]);
    a[2 * j + 1] = dot2(w, co, a[2 * j + 1]);
  }
  if (end) {
    *reinterpret_cast<u32x4*>(tile + tile_off(e)) =
        u32x4{pack_bf2(a[0], a[1]), pack_bf2(a[2], a[3]), pack_bf2(a[4], a[5]), pack_bf2(a[6], a[7])};
    const bool restart = e & kSlotEnd;
#pragma unroll
    for (int j = 0; j < 8; ++j) a[j] = restart ? 0.f : a[j];
  }
}

// Round-end bits of stream rows k0 .. k0+31 of a pair (bit i: row k0 + i ends a round).  Row
// mask words beyond the first come from the mask table (scalar loads: uniform address).
__device__ __forceinline__ unsigned chunk_ends(const int4& q, const unsigned* __restrict__ em, int k0) {
  if (k0 == 0) return (unsigned)q.w;
  const unsigned* w = em + q.z + (k0 >> 5);
  const unsigned long long m = (unsigned long long)w[0] | ((unsigned long long)w[1] << 32);
  return (unsigned)(m >> (k0 & 31));
}

// ---------------------------------------------------------------- forward stream chunks

struct FwdChunk {
  unsigned en[kCh];
  float cc[kCh];
};

// Load rows k0 .. k0+kCh-1 (k0 a multiple of 4) of a forward stream whose rows start at `off`
// (len >= 4, a multiple of 4): slot words and their coefficients, four rows per 16-byte load.
// Row groups past the stream's end re-read its last group and are skipped by fwd_compute.
__device__ __forceinline__ void fwd_load(const unsigned* __restrict__ st, int off, int len, int k0,
                                         const float* __restrict__ cv, int lane, FwdChunk& ch) {
#pragma unroll
  for (int g = 0; g < kCh / 4; ++g) {
    // a wave-uniform row base plus the lane's 16 bytes: scalar base, vector offset
    const long row = 64L * off + 256L * min(k0 / 4 + g, len / 4 - 1);
    const u32x4 w = gld(reinterpret_cast<const u32x4*>(st + row))[lane];
    const f32x4 c = gld(reinterpret_cast<const f32x4*>(cv + row))[lane];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      ch.en[4 * g + j] = w[j];
      ch.cc[4 * g + j] = c[j];
    }
  }
}

// The first n (uniform, a multiple of 4) slots of a loaded chunk, with their round-end bits;
// all kCh LDS rows are read first.
__device__ __forceinline__ void fwd_compute(const FwdChunk& ch, int n, unsigned ends, float scale,
                                            unsigned char* tile, float (&a)[8]) {
  u32x4 zv[kCh];
#pragma unroll
  for (int i = 0; i < kCh; ++i) zv[i] = lds_src(ch.en[i]);
#pragma unroll
  for (int i = 0; i < kCh; ++i) {
    if (i < n) {   // uniform
      unsigned ce, co;
      coef_words(ch.cc[i], scale, ce, co);
      accum_slot(ch.en[i], ce, co, zv[i], (ends >> i) & 1u, tile, a);
    }
  }
}

// ---------------------------------------------------------------- backward stream chunks

struct BwdEntries {
  unsigned en[kCh];   // slot words
};

// Rows k0 .. k0+kCh-1 of a backward stream (`st` = its first row, len a multiple of 4), four
// rows (32 bytes) per lane in two 16-byte loads; groups past the end re-read the last group.
__device__ __forceinline__ void bwd_load_entries(const unsigned* __restrict__ st, int len, int k0, int lane,
                                                 BwdEntries& ch) {
#pragma unroll
  for (int g = 0; g < kCh / 4; ++g) {
    const u32x4 w = gld(reinterpret_cast<const u32x4*>(st + 256L * min(k0 / 4 + g, len / 4 - 1)))[lane];
#pragma unroll
    for (int j = 0; j < 4; ++j) ch.en[4 * g + j] = w[j];
  }
}

// Coefficients of the same rows from the copy gathered into backward slot order (`cb` = the
// pair's first slot), one 16-byte load per 4-row group.
__device__ __forceinline__ void bwd_load_coeffs(const float* __restrict__ cb, int len, int k0, int lane,
                                                float (&cc)[kCh]) {
#pragma unroll
  for (int g = 0; g < kCh / 4; ++g) {
    const f32x4 c = gld(reinterpret_cast<const f32x4*>(cb + 256L * min(k0 / 4 + g, len / 4 - 1)))[lane];
#pragma unroll
    for (int j = 0; j < 4; ++j) cc[4 * g + j] = c[j];
  }
}

// This tile's share of dC / s for the rows of a chunk, written per 4-row group with one 16-byte
// store per lane to part (the pair's slots, k0 = the chunk's first stream row); groups past the
// stream's end (n = rows of the chunk inside it, a multiple of 4) write to the scratch row
// `trash`.  Padding slots write values the reduction never reads.
__device__ __forceinline__ void bwd_sddmm(const BwdEntries& ch, int n, int k0,
                                          const unsigned char* tile, float* __restrict__ part,
                                          float* __restrict__ trash, int lane) {
#pragma unroll
  for (int g = 0; g < kCh / 4; ++g) {
    f32x4 s4;
#pragma unroll
    for (int h = 0; h < 4; h += 2) {   // two slots' rows in flight at a time
      u32x4 uv[2], zv[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const unsigned e = ch.en[4 * g + h + i];
        uv[i] = lds_src(e);
        zv[i] = lds_at(tile, tile_off(e));
      }
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        float s = 0.f;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const unsigned uw = uv[i][j], zw = zv[i][j];
          s = dot2(uw, zw, s);
        }
        s4[h + i] = s;
      }
    }
    float* dst = 4 * g < n ? part + 256L * (k0 / 4 + g) + 4 * lane : trash + 4 * lane;
    *gst(reinterpret_cast<f32x4*>(dst)) = s4;
  }
}

__device__ __forceinline__ void bwd_spmm(const BwdEntries& ch, const float (&cc)[kCh], int n, unsigned ends,
                                         float scale, unsigned char* tile, float (&a)[8]) {
  constexpr int kH = kCh / 2;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    u32x4 uv[kH];
#pragma unroll
    for (int i = 0; i < kH; ++i) uv[i] = lds_src(ch.en[h * kH + i]);
#pragma unroll
    for (int i = 0; i < kH; ++i) {
      if (h * kH + i < n) {   // uniform
        unsigned ce, co;
        coef_words(cc[h * kH + i], scale, ce, co);
        accum_slot(ch.en[h * kH + i], ce, co, uv[i], (ends >> (h * kH + i)) & 1u, tile, a);
      }
    }
  }
}

struct FastArgs {
  const void* frag;   // synthesis fragments of the 128-wide block
  int T, nblk_in, nblk_out;
  const void* X;
  const void* const* Xs;
  long ldx;
  const void* G;
  const void* const* Gs;
  long ldg;
  void* Y;
  void* const* Ys;
  long ldy;
  const float* c;
  const float* const* cs;
  const float* cb;    // backward: coefficients in backward slot order, [batch][slots + 256]
  float* csave;       // forward: where to write that copy, [batch][slots + 256]
  const int* pos;     // per coefficient slot: its backward slot (padding: the scratch slot)
  int nslot;          // coefficient slots (>= 256 on this path)
  const int* bpad;    // backward slots with no entry: their copied coefficient is zero
  int nbpad;          // >= 1 (the scratch slot stands in when there is none)
  float scale, beta;
  int slots;          // dC partials per tile
  int pstride;        // floats per tile in the partial workspace: slots + a scratch row group
  float* partial;     // [batch][tile][pstride]
  long ntiles;
  // group calls: adapter blockIdx.y's own plan tables and workspace, and its token count
  // (device, clamped to [0, T]; NULL: T)
  const FastDesc* group;
  const int* tokens;
};

// Tokens of adapter bi in a group call (uniform in the workgroup).
__device__ __forceinline__ int group_tokens(const FastArgs& a, int bi) {
  const int t = a.tokens ? gld(a.tokens)[bi] : a.T;
  return max(0, min(t, a.T));
}

// s_waitcnt vmcnt(n) (n < 16), other counters untouched.
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 16, "vmcnt field");
  __builtin_amdgcn_s_waitcnt(0x0F70 | N);
}

// One 16-byte load per lane straight into LDS: lane l's bytes land at LDS address lds + 16 l
// (lds wave-uniform).  Written as assembly because the compiler, which cannot tell which LDS
// bytes such a load writes, would otherwise wait for every one of them before any LDS read;
// the readers wait for exactly the loads they need with vm_wait, and the compiler, not knowing
// these loads, can only over-count its own waits.
__device__ __forceinline__ void dma16(const FF_GLOBAL void* src, unsigned lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds) : "memory", "m0");
}

// The input rows of one pair (16 rows of 256 bytes: row n = 8 bs + t, token columns past the
// tile's end repeating its last token) loaded into the 4 KB at `dst` without passing through
// registers, each load covering four whole rows; row n keeps its 16-byte chunk c at position
// c ^ n.
__device__ __forceinline__ void dma_rows(const u16* rows, long ld, int nt, int blk0, int lane, unsigned char* dst) {
  const int pos = lane & 15;
  const unsigned base = (unsigned)(size_t)(__attribute__((address_space(3))) unsigned char*)dst;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 4 * i + (lane >> 4), t = min(r & 7, nt - 1), bs = r >> 3;
    dma16(gld(rows + (long)t * ld + (blk0 + bs) * kW + 8 * (pos ^ r)), base + 1024 * i);
  }
}

// The analysis operand of a pair staged by dma_rows: lane (column n, k-group g) takes chunk
// 4 ks + g of row n (inputs 32 ks + 8 g .. +7, as load_act would have loaded them).
__device__ __forceinline__ void read_rows(const unsigned char* src, int lane, u32x4 (&b)[kKT]) {
  const int n = lane & 15, g = lane >> 4;
#pragma unroll
  for (int ks = 0; ks < kKT; ++ks)
    b[ks] = *reinterpret_cast<const u32x4*>(src + n * 256 + (unsigned)(((4 * ks + g) ^ n) * 16));
}

// Analysis of every pair of blocks of a tile into a coefficient-major LDS array.  Each pair's
// inputs are staged in the pair's own 4 KB of the array, which its analysis overwrites only after
// reading them (a wave's LDS operations execute in order), two pairs ahead.  Loads for pairs past
// the end go to `spare` (the wave's free pair tile), so that every iteration issues the same
// loads and the counted waits stay exact; they are all waited for before returning.
__device__ __forceinline__ void analysis_phase(const Frag& F, const u16* rows, long ld, int nt, int np, int wave,
                                               int lane, unsigned char* lds, unsigned char* spare) {
  const int last = np - 1;
  const int n = lane & 15, q = lane >> 4;
  const unsigned off = ((q >> 1) * kW + n) * 16 + 8 * (q & 1);   // this lane's row of pair 0
  const unsigned sgn = (n & 1) ? 0x80008000u : 0u;               // odd coefficients negated
  constexpr unsigned kPairBytes = 2 * kW * kTT * 2;
  auto slot = [&](int p) { return p < np ? lds + p * kPairBytes : spare; };
  wave_lds_fence();
  dma_rows(rows, ld, nt, 2 * min(wave, last), lane, slot(wave));
  dma_rows(rows, ld, nt, 2 * min(wave + kWaves, last), lane, slot(wave + kWaves));
  issue_point();
  for (int p = wave; p < np; p += kWaves) {
    vm_wait<4>();   // this pair's four loads (the next pair's four may still be in flight)
    wave_lds_fence();
    u32x4 b[kKT];
    read_rows(slot(p), lane, b);
    wave_lds_fence();
    dma_rows(rows, ld, nt, 2 * min(p + 2 * kWaves, last), lane, slot(p + 2 * kWaves));
    issue_point();
    f32x4 acc[kMT];
    mfma_block_t(F, b, acc, ~0u);
    store_coef_t(lds + p * kPairBytes, off, acc, sgn);
  }
  vm_wait_all();
  wave_lds_fence();
}

// The stream tables are separate restrict-qualified arguments: the kernel never writes them,
// so their wave-uniform reads become scalar loads, which do not wait for vector stores.
// GROUP: adapter blockIdx.y runs its own plan (a.group) on its own token count; such calls keep
// no backward-ordered copy (the group backward writes its own).
template <bool BETA, bool GROUP>
__global__ void __launch_bounds__(kThreads, 2) fwd128(FastArgs a, const int4* __restrict__ pl,
                                                      const unsigned* __restrict__ fst,
                                                      const unsigned* __restrict__ em) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  unsigned char* zL = smem;                                        // n rows x 8 tokens x 2 bytes
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  unsigned char* tile = zL + (long)a.nblk_in * kW * kTT * 2 + wave * (2 * kW * kTT * 2);
  const int bi = blockIdx.y;
  if constexpr (GROUP) {
    const FastDesc* d = a.group + bi;
    pl = d->fwd_pl;
    fst = d->fwd_st;
    em = d->fwd_em;
    a.T = group_tokens(a, bi);
  }
  const int t0 = blockIdx.x * kTT, nt = min(kTT, a.T - t0);
  if (GROUP && nt <= 0) return;   // past this adapter's tokens (uniform)
  const u16* X = reinterpret_cast<const u16*>(a.Xs ? a.Xs[bi] : a.X) + (long)t0 * a.ldx;
  u16* Y = reinterpret_cast<u16*>(a.Ys ? a.Ys[bi] : a.Y) + (long)t0 * a.ldy;
  const float* cv = a.cs ? a.cs[bi] : a.c;
  const int npo = a.nblk_out / 2, lastp = npo - 1;

  // This workgroup's share of the coefficient copy in the backward's slot order: coefficient
  // slots, then the backward's padding slots (zero).  Read first, written after the analysis;
  // every lane loads and stores (lanes past the share repeat its last item, an identical write).
  const int nitem = GROUP ? 0 : a.nslot + a.nbpad;
  const int per = (nitem + (int)gridDim.x - 1) / (int)gridDim.x;
  const int j0 = (int)blockIdx.x * per, jn = min(nitem, j0 + per);
  int spos = 0;
  float sval = 0.f;
  float* csave = nullptr;
  if constexpr (!GROUP) {
    const int js = max(min(j0 + (int)threadIdx.x, jn - 1), 0);
    const bool is_coef = js < a.nslot;
    const int pc = gld(a.pos)[min(js, a.nslot - 1)], pp = gld(a.bpad)[min(max(js - a.nslot, 0), a.nbpad - 1)];
    const float cval = gld(cv)[min(js, a.nslot - 1)];
    spos = is_coef ? pc : pp;
    sval = is_coef ? cval : 0.f;
    csave = a.csave + (long)bi * (a.slots + 256);
  }

  u32x4 fr[kFragPerThread];
  frag_fetch(a.frag, fr);
  issue_point();
  // first stream chunk of this wave's first output pair, in flight during the analysis; the
  // pair entries run one pair ahead of the chunks, so their scalar loads are never waited on
  // at a pair's start
  int4 q = pl[min(wave, lastp)];
  int4 qn = pl[min(wave + kWaves, lastp)];
  FwdChunk ch;
  fwd_load(fst, q.x, q.y, 0, cv, lane, ch);
  issue_point();

  Frag F;
  frag_stage(fr, reinterpret_cast<u32x4*>(smem), lane, F);
  analysis_phase(F, X, a.ldx, nt, a.nblk_in / 2, wave, lane, zL, tile);
  if constexpr (!GROUP) gst(csave)[spos] = sval;
  __syncthreads();

  // One output pair: its chunk is in `cur`; the next pair's chunk is loaded into `nxt` first,
  // a whole pair ahead of its use.  The loop runs two pairs per iteration with the buffers'
  // roles swapped, so no chunk is ever copied between registers.
  const int steps = (npo - wave + kWaves - 1) / kWaves;
  // A pair's synthesis is stored at the start of the wave's next pair, after that pair's
  // stream loads: the loads do not queue behind the stores, and the MFMA results are waited
  // for a whole sparse phase later.
  // The wave's first pair is a separate instance with no store, so that every other instance
  // stores unconditionally and the compiler's memory counters stay exact (a store that may or
  // may not have been issued makes it wait for all of them).
  f32x4 acc[kMT];
  auto pair = [&](int p, FwdChunk& cur, FwdChunk& nxt, auto first) {
    prio_by_progress((p - wave) / kWaves, steps);
    fwd_load(fst, qn.x, qn.y, 0, cv, lane, nxt);
    const int4 qnn = pl[min(p + 2 * kWaves, lastp)];
    issue_point();
    if constexpr (!decltype(first)::value) store_act<BETA>(Y, a.ldy, nt, 2 * (p - kWaves), lane, acc, a.beta, tile);
    // v = C z for this pair into the tile
    const int off = q.x, len = q.y;
    zero_tile(tile, lane);
    float acc8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    fwd_compute(cur, min(kCh, len), (unsigned)q.w, a.scale, tile, acc8);
    if (len > kCh) {   // long stream
      for (int k0 = kCh; k0 < len; k0 += kCh) {
        fwd_load(fst, off, len, k0, cv, lane, cur);
        fwd_compute(cur, min(kCh, len - k0), chunk_ends(q, em, k0), a.scale, tile, acc8);
      }
      vm_wait_all();
    }
    wave_lds_fence();
    // y = beta y + s P_out v
    u32x4 b[kKT];
    load_tile_act(tile, lane, b);
    wave_lds_fence();
    mfma_block(F, b, acc);
    q = qn;
    qn = qnn;
  };
  FwdChunk ch2;
  if (wave < npo) {
    const std::true_type first;
    const std::false_type later;
    int plast = wave;
    pair(wave, ch, ch2, first);
    if (wave + kWaves < npo) {
      pair(wave + kWaves, ch2, ch, later);
      plast = wave + kWaves;
    }
    for (int p = wave + 2 * kWaves; p < npo; p += 2 * kWaves) {
      pair(p, ch, ch2, later);
      plast = p;
      if (p + kWaves < npo) {
        pair(p + kWaves, ch2, ch, later);
        plast = p + kWaves;
      }
    }
    store_act<BETA>(Y, a.ldy, nt, 2 * plast, lane, acc, a.beta, tile);
  }
  // shares longer than one slot per thread (grids of few tiles)
  if (!GROUP && per > kThreads)
    for (int j = j0 + kThreads + (int)threadIdx.x; j < jn; j += kThreads) {
      if (j < a.nslot)
        gst(csave)[gld(a.pos)[j]] = gld(cv)[j];
      else
        gst(csave)[gld(a.bpad)[j - a.nslot]] = 0.f;
    }
}

template <bool DX, bool DC, bool BETA, bool GROUP>
__global__ void __launch_bounds__(kThreads, 2) bwd128(FastArgs a, const int4* __restrict__ pl,
                                                      const unsigned* __restrict__ bst,
                                                      const unsigned* __restrict__ em) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  unsigned char* uL = smem;                                        // m rows x 8 tokens x 2 bytes
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  unsigned char* tile = uL + (long)a.nblk_out * kW * kTT * 2 + wave * (2 * kW * kTT * 2);
  const int bi = blockIdx.y;
  long tile_row = (long)bi * a.ntiles + blockIdx.x;   // this tile's dC partial row
  if constexpr (GROUP) {   // the adapter's own plan, workspace (batch slot 0) and tokens
    const FastDesc* d = a.group + bi;
    if (d->bwd16) return;   // served by the 16-token kernel of the same call
    pl = d->bwd_pl;
    bst = d->bwd_st;
    em = d->bwd_em;
    a.slots = d->slots;
    a.pstride = d->slots + 256;
    a.cb = d->coef;
    a.partial = d->partial;
    a.T = group_tokens(a, bi);
    tile_row = blockIdx.x;
  }
  const int t0 = blockIdx.x * kTT, nt = min(kTT, a.T - t0);
  if (GROUP && nt <= 0) return;   // past this adapter's tokens (uniform)
  const u16* G = reinterpret_cast<const u16*>(a.Gs ? a.Gs[bi] : a.G) + (long)t0 * a.ldg;
  const u16* X = DC ? reinterpret_cast<const u16*>(a.Xs ? a.Xs[bi] : a.X) + (long)t0 * a.ldx : nullptr;
  u16* dX = DX ? reinterpret_cast<u16*>(a.Ys ? a.Ys[bi] : a.Y) + (long)t0 * a.ldy : nullptr;
  const float* cbw = DX ? a.cb + (GROUP ? 0L : (long)bi * (a.slots + 256)) : nullptr;
  float* part = DC ? a.partial + tile_row * a.pstride : nullptr;
  float* trash = DC ? part + a.slots : nullptr;
  // dC sums only over the tile's tokens: activation columns past its end are zeroed
  const unsigned km = (lane & 7) < nt ? ~0u : 0u;
  // this lane's place in the pair tile for the analysis of x
  const unsigned zoff = tile_lane_off(lane);
  const unsigned zsgn = (lane & 1) ? 0x80008000u : 0u;
  const int npi = a.nblk_in / 2, lastp = npi - 1;

  u32x4 fr[kFragPerThread];
  frag_fetch(a.frag, fr);
  issue_point();
  // this wave's first input pair: stream entries and x in flight during the analysis of g
  int4 q = pl[min(wave, lastp)];
  BwdEntries ch;
  bwd_load_entries(bst + (long)q.x * 64, q.y, 0, lane, ch);
  u32x4 bx[kKT];
  if (DC) load_act(X, a.ldx, nt, 2 * min(wave, lastp), lane, bx);
  issue_point();

  Frag F;
  frag_stage(fr, reinterpret_cast<u32x4*>(smem), lane, F);
  analysis_phase(F, G, a.ldg, nt, a.nblk_out / 2, wave, lane, uL, tile);
  __syncthreads();

  // Two passes over this wave's input pairs, so that each holds few registers: dC, then dX.
  const int npw = (npi - wave + kWaves - 1) / kWaves;   // this wave's pairs per pass
  const int steps = (DC ? npw : 0) + (DX ? npw : 0);
  if (DC) {
    // one input pair; the next pair's entries are loaded into `nxt` a whole pair ahead of
    // their use, two pairs per iteration with the buffers' roles swapped
    auto pair = [&](int p, BwdEntries& ch, BwdEntries& chn) {
      prio_by_progress((p - wave) / kWaves, steps);
      const int len = q.y;
      const unsigned* st = bst + (long)q.x * 64;
      const int4 qn = pl[min(p + kWaves, lastp)];
      bwd_load_entries(bst + (long)qn.x * 64, qn.y, 0, lane, chn);
      issue_point();
      // z = P_in^T x for this pair (tile columns past the tile's end zeroed), then this
      // tile's share of dC
      {
        f32x4 acc[kMT];
        mfma_block_t(F, bx, acc, km);
        store_tile_t(tile, zoff, acc, zsgn);
      }
      wave_lds_fence();
      load_act(X, a.ldx, nt, 2 * min(p + kWaves, lastp), lane, bx);
      issue_point();
      float* pp = part + (long)q.x * 64;
      bwd_sddmm(ch, min(kCh, len), 0, tile, pp, trash, lane);
      if (len > kCh) {   // long stream
        for (int k0 = kCh; k0 < len; k0 += kCh) {
          BwdEntries ck;
          bwd_load_entries(st, len, k0, lane, ck);
          bwd_sddmm(ck, min(kCh, len - k0), k0, tile, pp, trash, lane);
        }
        vm_wait_all();
      }
      wave_lds_fence();
      q = qn;
    };
    BwdEntries ch2;
    for (int p = wave; p < npi; p += 2 * kWaves) {
      pair(p, ch, ch2);
      if (p + kWaves < npi) pair(p + kWaves, ch2, ch);
    }
    if (DX) {   // restart at this wave's first pair
      q = pl[min(wave, lastp)];
      bwd_load_entries(bst + (long)q.x * 64, q.y, 0, lane, ch);
    }
  }
  if (DX) {
    float cc[kCh], cc2[kCh];
    bwd_load_coeffs(cbw + (long)q.x * 64, q.y, 0, lane, cc);
    // one input pair; the next pair's entries and coefficients are loaded at its start, two
    // pairs per iteration with the buffers' roles swapped
    auto pair = [&](int p, BwdEntries& ch, float (&cc)[kCh], BwdEntries& chn, float (&ccn)[kCh]) {
      prio_by_progress((DC ? npw : 0) + (p - wave) / kWaves, steps);
      const int len = q.y;
      const unsigned* st = bst + (long)q.x * 64;
      const float* cbp = cbw + (long)q.x * 64;
      const int4 qn = pl[min(p + kWaves, lastp)];
      bwd_load_entries(bst + (long)qn.x * 64, qn.y, 0, lane, chn);
      bwd_load_coeffs(cbw + (long)qn.x * 64, qn.y, 0, lane, ccn);
      issue_point();
      // q = C^T u for this pair, then dX = beta dX + s P_in q
      zero_tile(tile, lane);
      float acc8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      bwd_spmm(ch, cc, min(kCh, len), (unsigned)q.w, a.scale, tile, acc8);
      if (len > kCh) {   // long stream
        for (int k0 = kCh; k0 < len; k0 += kCh) {
          BwdEntries ck;
          float ckc[kCh];
          bwd_load_entries(st, len, k0, lane, ck);
          bwd_load_coeffs(cbp, len, k0, lane, ckc);
          bwd_spmm(ck, ckc, min(kCh, len - k0), chunk_ends(q, em, k0), a.scale, tile, acc8);
        }
        vm_wait_all();
      }
      wave_lds_fence();
      u32x4 b[kKT];
      f32x4 acc[kMT];
      load_tile_act(tile, lane, b);
      wave_lds_fence();
      mfma_block(F, b, acc);
      store_act<BETA>(dX, a.ldy, nt, 2 * p, lane, acc, a.beta, tile);
      q = qn;
    };
    BwdEntries ch2;
    for (int p = wave; p < npi; p += 2 * kWaves) {
      pair(p, ch, cc, ch2, cc2);
      if (p + kWaves < npi) pair(p + kWaves, ch2, cc2, ch, cc);
    }
  }
}

// ---------------------------------------------------------------- 16-token backward
//
// The same backward for 16 tokens per workgroup (8 waves, one workgroup per CU), used when the
// output side's coefficient array for 16 tokens fits in LDS next to the wave tiles (m <= 4096)
// and every backward stream has at most 16 rows.  The array has rows of 32 bytes (both token
// halves of a coefficient), the slot words' source field addresses them, and each pair's stream
// is loaded once and applied to the two 8-token halves in turn through the same 4 KB tile
// layout, so that a stream's slot words, coefficients and dC partial sums serve 16 tokens: half
// the partial sums to write and reduce, and half the stream loads per token.
constexpr int kTT16 = 16;
constexpr int kWaves16 = 8;
constexpr int kThreads16 = 64 * kWaves16;
constexpr int kCh16 = 16;   // a whole stream held in registers

// Store the result of mfma_block_t for token half h into a coefficient-major array of 32-byte
// rows, half h of row c at bytes 16 (h ^ (c & 1)) of the row, so that the 16-byte reads of one
// half at random rows spread over all banks: `row` is this lane's byte offset in row tile 0 for
// its half (odd coefficients negated).
__device__ __forceinline__ void store_coef16_t(unsigned char* lds, unsigned row, const f32x4 (&acc)[kMT],
                                               unsigned sgn) {
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt) {
    const unsigned w0 = pack_bf2(acc[mt][0], acc[mt][1]) ^ sgn, w1 = pack_bf2(acc[mt][2], acc[mt][3]) ^ sgn;
    *reinterpret_cast<u32x2*>(lds + row + 512 * mt) = u32x2{w0, w1};
  }
}

// Analysis of both token halves of every pair into the 32-byte-row array.  A pair's 8 KB stage
// both halves' inputs (4 KB each), which are read before either half's result is written over
// them; pairs run two ahead and every wait counts exactly the loads issued after it.  Tokens
// 8..15 of a tile with at most 8 tokens repeat tokens 0..7 (their results are never used).
__device__ __forceinline__ void analysis16(const Frag& F, const u16* rows, long ld, int nt, int np, int wave,
                                           int lane, unsigned char* lds) {
  const int n = lane & 15, q = lane >> 4;
  // this lane's coefficient (16 mt + n of block q >> 1) has the parity of n
  const unsigned off0 = ((q >> 1) * kW + n) * 32 + 8 * (q & 1) + 16 * (n & 1), off1 = off0 ^ 16;
  const unsigned sgn = (n & 1) ? 0x80008000u : 0u;
  constexpr unsigned kPair = 2 * kW * 32;
  const u16* rows1 = nt > 8 ? rows + 8 * ld : rows;
  const int nt0 = min(nt, 8), nt1 = nt > 8 ? nt - 8 : nt0;
  auto issue = [&](int p) {
    dma_rows(rows, ld, nt0, 2 * p, lane, lds + p * kPair);
    dma_rows(rows1, ld, nt1, 2 * p, lane, lds + p * kPair + 4096);
  };
  wave_lds_fence();
  if (wave < np) issue(wave);
  if (wave + kWaves16 < np) issue(wave + kWaves16);
  issue_point();
  for (int p = wave; p < np; p += kWaves16) {
    if (p + kWaves16 < np)
      vm_wait<8>();   // this pair's eight loads (the next pair's eight may still be in flight)
    else
      vm_wait<0>();
    wave_lds_fence();
    u32x4 b0[kKT], b1[kKT];
    read_rows(lds + p * kPair, lane, b0);
    read_rows(lds + p * kPair + 4096, lane, b1);
    wave_lds_fence();
    if (p + 2 * kWaves16 < np) issue(p + 2 * kWaves16);
    issue_point();
    f32x4 acc[kMT];
    mfma_block_t(F, b0, acc, ~0u);
    store_coef16_t(lds + p * kPair, off0, acc, sgn);
    mfma_block_t(F, b1, acc, ~0u);
    store_coef16_t(lds + p * kPair, off1, acc, sgn);
  }
  wave_lds_fence();
}

// Token half h (h16 = 16 h) of the uL row of a slot word, whose source field already holds the
// row's half 0 (at 16 (c & 1) within row c).
__device__ __forceinline__ u32x4 lds_src16(unsigned e, unsigned h16) {
  return *(const __attribute__((address_space(3))) u32x4*)(size_t)((e & kSlotSrcMask) ^ h16);
}

// A whole backward stream (len <= 16, a multiple of 4): slot words, four rows per 16-byte load;
// groups past the end re-read the last group.
__device__ __forceinline__ void bwd16_entries(const unsigned* __restrict__ st, int len, int lane,
                                              unsigned (&en)[kCh16]) {
#pragma unroll
  for (int g = 0; g < kCh16 / 4; ++g) {
    const u32x4 w = gld(reinterpret_cast<const u32x4*>(st + 256L * min(g, len / 4 - 1)))[lane];
#pragma unroll
    for (int j = 0; j < 4; ++j) en[4 * g + j] = w[j];
  }
}

__device__ __forceinline__ void bwd16_coeffs(const float* __restrict__ cb, int len, int lane, float (&cc)[kCh16]) {
#pragma unroll
  for (int g = 0; g < kCh16 / 4; ++g) {
    const f32x4 c = gld(reinterpret_cast<const f32x4*>(cb + 256L * min(g, len / 4 - 1)))[lane];
#pragma unroll
    for (int j = 0; j < 4; ++j) cc[4 * g + j] = c[j];
  }
}

// s[i] (+)= sum over the half's 8 tokens of u[a_i] z[b_i] for the first n slots (uniform), four
// slots' rows in flight at a time.
template <bool FIRST>
__device__ __forceinline__ void sddmm16(const unsigned (&en)[kCh16], int n, const unsigned char* tile, unsigned h16,
                                        float (&s)[kCh16]) {
#pragma unroll
  for (int g = 0; g < kCh16 / 4; ++g) {
    if (4 * g < n) {   // uniform
      u32x4 uv[4], zv[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const unsigned e = en[4 * g + i];
        uv[i] = lds_src16(e, h16);
        zv[i] = lds_at(tile, tile_off(e));
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float d = FIRST ? 0.f : s[4 * g + i];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const unsigned uw = uv[i][j], zw = zv[i][j];
          d = dot2(uw, zw, d);
        }
        s[4 * g + i] = d;
      }
    }
  }
}

// q = C^T u for token half h over the first n slots into the tile (round ends as in accum_slot).
__device__ __forceinline__ void spmm16(const unsigned (&en)[kCh16], const float (&cc)[kCh16], int n, unsigned ends,
                                       float scale, unsigned h16, unsigned char* tile, float (&a)[8]) {
  constexpr int kH = kCh16 / 2;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    if (h * kH < n) {   // uniform
      u32x4 uv[kH];
#pragma unroll
      for (int i = 0; i < kH; ++i) uv[i] = lds_src16(en[h * kH + i], h16);
#pragma unroll
      for (int i = 0; i < kH; ++i) {
        if (h * kH + i < n) {   // uniform
          unsigned ce, co;
          coef_words(cc[h * kH + i], scale, ce, co);
          accum_slot(en[h * kH + i], ce, co, uv[i], (ends >> (h * kH + i)) & 1u, tile, a);
        }
      }
    }
  }
}

template <bool DX, bool DC, bool BETA, bool GROUP>
__global__ void __launch_bounds__(kThreads16, 1) bwd16(FastArgs a, const int4* __restrict__ pl,
                                                       const unsigned* __restrict__ bst) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  unsigned char* uL = smem;   // m rows x 16 tokens x 2 bytes
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  unsigned char* tile = uL + (long)a.nblk_out * kW * kTT16 * 2 + wave * (2 * kW * kTT * 2);
  const int bi = blockIdx.y;
  long tile_row = (long)bi * a.ntiles + blockIdx.x;   // this tile's dC partial row
  if constexpr (GROUP) {   // the adapter's own plan, workspace (batch slot 0) and tokens
    const FastDesc* d = a.group + bi;
    if (!d->bwd16) return;   // served by the 8-token kernel of the same call
    pl = d->bwd_pl;
    bst = d->bwd_st;
    a.slots = d->slots;
    a.pstride = d->slots + 256;
    a.cb = d->coef;
    a.partial = d->partial;
    a.T = group_tokens(a, bi);
    tile_row = blockIdx.x;
  }
  const int t0 = blockIdx.x * kTT16, nt = min(kTT16, a.T - t0);
  if (GROUP && nt <= 0) return;   // past this adapter's tokens (uniform)
  const bool two = nt > 8;   // the tile has a second token half
  const int nt0 = min(nt, 8), nt1 = two ? nt - 8 : nt0;
  const u16* G = reinterpret_cast<const u16*>(a.Gs ? a.Gs[bi] : a.G) + (long)t0 * a.ldg;
  const u16* X0 = DC ? reinterpret_cast<const u16*>(a.Xs ? a.Xs[bi] : a.X) + (long)t0 * a.ldx : nullptr;
  const u16* X1 = DC ? (two ? X0 + 8 * a.ldx : X0) : nullptr;
  u16* dX0 = DX ? reinterpret_cast<u16*>(a.Ys ? a.Ys[bi] : a.Y) + (long)t0 * a.ldy : nullptr;
  u16* dX1 = DX ? dX0 + 8 * a.ldy : nullptr;   // stored only when the tile has a second half
  const float* cbw = DX ? a.cb + (GROUP ? 0L : (long)bi * (a.slots + 256)) : nullptr;
  float* part = DC ? a.partial + tile_row * a.pstride : nullptr;
  float* trash = DC ? part + a.slots : nullptr;
  // dC sums only over the tile's tokens: activation columns past its end are zeroed
  const unsigned km0 = (lane & 7) < nt ? ~0u : 0u, km1 = (lane & 7) + 8 < nt ? ~0u : 0u;
  const unsigned zoff = tile_lane_off(lane);
  const unsigned zsgn = (lane & 1) ? 0x80008000u : 0u;
  const int npi = a.nblk_in / 2, lastp = npi - 1;

  u32x4 fr[frag_per_thread<kThreads16>()];
  frag_fetch<kThreads16>(a.frag, fr);
  issue_point();
  int4 q = pl[min(wave, lastp)];
  unsigned en[kCh16];
  bwd16_entries(bst + (long)q.x * 64, q.y, lane, en);
  u32x4 bx0[kKT], bx1[kKT];
  if (DC) {
    load_act(X0, a.ldx, nt0, 2 * min(wave, lastp), lane, bx0);
    load_act(X1, a.ldx, nt1, 2 * min(wave, lastp), lane, bx1);
  }
  issue_point();

  Frag F;
  frag_stage<kThreads16>(fr, reinterpret_cast<u32x4*>(smem), lane, F);
  analysis16(F, G, a.ldg, nt, a.nblk_out / 2, wave, lane, uL);
  __syncthreads();

  const int npw = (npi - wave + kWaves16 - 1) / kWaves16;
  const int steps = (DC ? npw : 0) + (DX ? npw : 0);
  if (DC) {
    auto pair = [&](int p, unsigned (&ch)[kCh16], unsigned (&chn)[kCh16]) {
      prio_by_progress((p - wave) / kWaves16, steps);
      const int len = q.y;
      const int4 qn = pl[min(p + kWaves16, lastp)];
      bwd16_entries(bst + (long)qn.x * 64, qn.y, lane, chn);
      issue_point();
      float sd[kCh16];
      {
        f32x4 acc[kMT];
        mfma_block_t(F, bx0, acc, km0);
        store_tile_t(tile, zoff, acc, zsgn);
      }
      wave_lds_fence();
      load_act(X0, a.ldx, nt0, 2 * min(p + kWaves16, lastp), lane, bx0);
      issue_point();
      sddmm16<true>(ch, len, tile, 0u, sd);
      wave_lds_fence();
      {   // the second half (all columns masked when the tile has no second half)
        f32x4 acc[kMT];
        mfma_block_t(F, bx1, acc, km1);
        store_tile_t(tile, zoff, acc, zsgn);
        wave_lds_fence();
        sddmm16<false>(ch, len, tile, 16u, sd);
        wave_lds_fence();
      }
      load_act(X1, a.ldx, nt1, 2 * min(p + kWaves16, lastp), lane, bx1);
      issue_point();
      float* pp = part + (long)q.x * 64;
#pragma unroll
      for (int g = 0; g < kCh16 / 4; ++g) {
        float* dst = 4 * g < len ? pp + 256L * g + 4 * lane : trash + 4 * lane;
        *gst(reinterpret_cast<f32x4*>(dst)) = f32x4{sd[4 * g], sd[4 * g + 1], sd[4 * g + 2], sd[4 * g + 3]};
      }
      q = qn;
    };
    unsigned en2[kCh16];
    for (int p = wave; p < npi; p += 2 * kWaves16) {
      pair(p, en, en2);
      if (p + kWaves16 < npi) pair(p + kWaves16, en2, en);
    }
    if (DX) {   // restart at this wave's first pair
      q = pl[min(wave, lastp)];
      bwd16_entries(bst + (long)q.x * 64, q.y, lane, en);
    }
  }
  if (DX) {
    float cc[kCh16], cc2[kCh16];
    bwd16_coeffs(cbw + (long)q.x * 64, q.y, lane, cc);
    auto pair = [&](int p, unsigned (&ch)[kCh16], float (&cv)[kCh16], unsigned (&chn)[kCh16],
                    float (&cvn)[kCh16]) {
      prio_by_progress((DC ? npw : 0) + (p - wave) / kWaves16, steps);
      const int len = q.y;
      const int4 qn = pl[min(p + kWaves16, lastp)];
      bwd16_entries(bst + (long)qn.x * 64, qn.y, lane, chn);
      bwd16_coeffs(cbw + (long)qn.x * 64, qn.y, lane, cvn);
      issue_point();
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        zero_tile(tile, lane);
        float acc8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        spmm16(ch, cv, len, (unsigned)q.w, a.scale, 16u * h, tile, acc8);
        wave_lds_fence();
        u32x4 b[kKT];
        f32x4 acc[kMT];
        load_tile_act(tile, lane, b);
        wave_lds_fence();
        mfma_block(F, b, acc);
        // (a tile without a second half computes one from repeated inputs and drops it; only the
        // following pair's first wait counts the skipped stores, next to loads issued with them)
        if (h == 0 || two) store_act<BETA>(h ? dX1 : dX0, a.ldy, h ? nt1 : nt0, 2 * p, lane, acc, a.beta, tile);
      }
      q = qn;
    };
    unsigned en2[kCh16];
    for (int p = wave; p < npi; p += 2 * kWaves16) {
      pair(p, en, cc, en2, cc2);
      if (p + kWaves16 < npi) pair(p + kWaves16, en2, cc2, en, cc);
    }
  }
}

// cb[batch][pos[j]] = c[batch][j]: the backward's coefficients scattered into its own stream
// order (one coalesced load per coefficient, no dependent load), so that it loads them like the
// forward does.  Padding slots go to a scratch slot past the backward slots.
__global__ void __launch_bounds__(256) scatter_bwd_coef(const float* c, const float* const* cs,
                                                        const int* __restrict__ pos, int nslot,
                                                        const int* __restrict__ bpad, int nbpad, int cstride,
                                                        float* cb) {
  const int bi = blockIdx.y;
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= nslot + nbpad) return;
  if (j < nslot) {
    const float* cv = cs ? cs[bi] : c;
    gst(cb)[(long)bi * cstride + gld(pos)[j]] = gld(cv)[j];
  } else {
    gst(cb)[(long)bi * cstride + gld(bpad)[j - nslot]] = 0.f;   // padding of the backward order
  }
}

// p[0 .. n) = 0 (a fill kernel rather than a memset node, so that captured graphs replay it).
__global__ void __launch_bounds__(256) fill_zero(float* p, int n) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j < n) gst(p)[j] = 0.f;
}

// dC[j] = [dC[j] +] s * sum_tiles partial[tile][slot] for every valid slot of the backward
// streams (j = the slot's coefficient slot).  A workgroup owns 64 backward slots; each of its
// 16 waves sums 1/16 of the tiles with all loads of a pass in flight, and the 16 sums are
// combined in a fixed order.  Blocks past the reduction blocks zero the padding slots of dC
// (overwrite mode only).
constexpr int kRedWaves = 16;
constexpr int kRedBatch = 8;

__global__ void __launch_bounds__(64 * kRedWaves) reduce128(const float* __restrict__ partial, long ntiles,
                                                            int slots, int pstride, const unsigned* __restrict__ dst,
                                                            float scale, int accumulate, float* dC,
                                                            float* const* dCs, const int* __restrict__ pad,
                                                            int npad, int nred) {
  __shared__ float red[kRedWaves][64];
  const int bi = blockIdx.y;
  float* out = dCs ? dCs[bi] : dC;
  if ((int)blockIdx.x >= nred) {
    const int i = ((int)blockIdx.x - nred) * 64 * kRedWaves + (int)threadIdx.x;
    if (i < npad) gst(out)[gld(pad)[i]] = 0.f;
    return;
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int slot = blockIdx.x * 64 + lane;
  float s = 0.f;
  if (slot < slots) {
    const float* p = partial + (long)bi * ntiles * pstride + slot;
    for (long t0 = w; t0 < ntiles; t0 += (long)kRedWaves * kRedBatch) {
      float v[kRedBatch];
#pragma unroll
      for (int j = 0; j < kRedBatch; ++j) {
        const long t = t0 + (long)j * kRedWaves;
        v[j] = t < ntiles ? gld(p)[t * pstride] : 0.f;
      }
#pragma unroll
      for (int j = 0; j < kRedBatch; ++j) s += v[j];
    }
  }
  red[w][lane] = s;
  __syncthreads();
  if (w == 0 && slot < slots) {
    float tot = 0.f;
#pragma unroll
    for (int i = 0; i < kRedWaves; ++i) tot += red[i][lane];
    const unsigned j = gld(dst)[slot];   // the slot's coefficient slot, or ~0 for padding
    if (j != ~0u) {
      const float v = scale * tot;
      gst(out)[j] = accumulate ? gld(out)[j] + v : v;
    }
  }
}

// Group calls: scatter_bwd_coef with every adapter's own plan (its copy cleared first, since
// its over-read margin may hold another plan's values).
__global__ void __launch_bounds__(256) scatter_bwd_coef_group(const float* const* cs, const FastDesc* group) {
  const int bi = blockIdx.y;
  const FastDesc* d = group + bi;
  const int nslot = d->coef_slots, nbpad = d->nbpad;
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= nslot + nbpad) return;
  if (j < nslot)
    gst(d->coef)[gld(d->bwd_pos)[j]] = gld(cs[bi])[j];
  else
    gst(d->coef)[gld(d->bwd_pad)[j - nslot]] = 0.f;
}

__global__ void __launch_bounds__(256) clear_copy_group(const FastDesc* group) {
  const FastDesc* d = group + blockIdx.y;
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j < d->slots + 256) gst(d->coef)[j] = 0.f;
}

// Group calls: reduce128 over each adapter's own tiles (its token count / tt of them), slots and
// destinations; blocks past an adapter's share return.
__global__ void __launch_bounds__(64 * kRedWaves) reduce128_group(const FastDesc* group, const int* tokens, int T,
                                                                  float scale, int accumulate, float* const* dCs) {
  __shared__ float red[kRedWaves][64];
  const int bi = blockIdx.y;
  const FastDesc* d = group + bi;
  float* out = dCs[bi];
  const int slots = d->slots, pstride = d->slots + 256;
  const int nred = (slots + 63) / 64;
  const int npad = accumulate ? 0 : d->npad;
  const int Tb = tokens ? max(0, min(gld(tokens)[bi], T)) : T;
  const int tt = d->bwd16 ? kTT16 : kTT;
  const long ntiles = (Tb + tt - 1) / tt;
  if ((int)blockIdx.x >= nred) {
    const int i = ((int)blockIdx.x - nred) * 64 * kRedWaves + (int)threadIdx.x;
    if (i < npad) gst(out)[gld(d->pad)[i]] = 0.f;
    return;
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int slot = blockIdx.x * 64 + lane;
  float s = 0.f;
  if (slot < slots) {
    const float* p = d->partial + slot;
    for (long t0 = w; t0 < ntiles; t0 += (long)kRedWaves * kRedBatch) {
      float v[kRedBatch];
#pragma unroll
      for (int j = 0; j < kRedBatch; ++j) {
        const long t = t0 + (long)j * kRedWaves;
        v[j] = t < ntiles ? gld(p)[t * pstride] : 0.f;
      }
#pragma unroll
      for (int j = 0; j < kRedBatch; ++j) s += v[j];
    }
  }
  red[w][lane] = s;
  __syncthreads();
  if (w == 0 && slot < slots) {
    float tot = 0.f;
#pragma unroll
    for (int i = 0; i < kRedWaves; ++i) tot += red[i][lane];
    const unsigned j = gld(d->bwd_dst)[slot];
    if (j != ~0u) {
      const float v = scale * tot;
      gst(out)[j] = accumulate ? gld(out)[j] + v : v;
    }
  }
}

void rec(hipEvent_t ev, hipStream_t s) {
  if (ev) (void)hipEventRecord(ev, s);
}

template <typename K>
hipError_t allow_lds(K* kernel) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel), hipFuncAttributeMaxDynamicSharedMemorySize,
                             kMaxLdsBytes);
}

}  // namespace

hipError_t configure_fast128() {
  static hipError_t once = [] {
    hipError_t e = hipSuccess;
    const hipError_t r[] = {allow_lds(&fwd128<false, false>),       allow_lds(&fwd128<true, false>),
                            allow_lds(&bwd128<true, true, false, false>), allow_lds(&bwd128<true, true, true, false>),
                            allow_lds(&bwd128<true, false, false, false>), allow_lds(&bwd128<true, false, true, false>),
                            allow_lds(&bwd128<false, true, false, false>), allow_lds(&bwd16<true, true, false, false>),
                            allow_lds(&bwd16<true, true, true, false>),   allow_lds(&bwd16<true, false, false, false>),
                            allow_lds(&bwd16<true, false, true, false>),  allow_lds(&bwd16<false, true, false, false>),
                            allow_lds(&fwd128<false, true>),        allow_lds(&fwd128<true, true>),
                            allow_lds(&bwd128<true, true, false, true>), allow_lds(&bwd128<true, true, true, true>),
                            allow_lds(&bwd128<true, false, false, true>), allow_lds(&bwd128<true, false, true, true>),
                            allow_lds(&bwd128<false, true, false, true>), allow_lds(&bwd16<true, true, false, true>),
                            allow_lds(&bwd16<true, true, true, true>),   allow_lds(&bwd16<true, false, false, true>),
                            allow_lds(&bwd16<true, false, true, true>),  allow_lds(&bwd16<false, true, false, true>)};
    for (hipError_t x : r)
      if (x != hipSuccess) e = x;
    return e;
  }();
  return once;
}

// The coefficient array (nblk 128-row blocks of 16 bytes) plus one 4 KB tile per wave; at least
// the 16 KB of fragments staged at kernel start.
size_t fast128_lds_bytes(int nblk) {
  const size_t b = (size_t)nblk * kW * kTT * 2 + (size_t)kWaves * 2 * kW * kTT * 2;
  const size_t frag = (size_t)kHT * kKT * 64 * 16;
  return b < frag ? frag : b;
}

size_t fast128_partial_floats(size_t bwd_slots) { return bwd_slots + 256; }

// The 16-token backward: the output side's array of 32-byte rows plus eight 4 KB wave tiles.
size_t fast16_lds_bytes(int nblk_out) {
  const size_t b = (size_t)nblk_out * kW * kTT16 * 2 + (size_t)kWaves16 * 2 * kW * kTT * 2;
  const size_t frag = (size_t)kHT * kKT * 64 * 16;
  return b < frag ? frag : b;
}

hipError_t launch_fwd128(const ff_plan* p, int count, int T, ActPtrs X, int64_t ldx, const float* c,
                         const float* const* cs, float scale, float beta, ActPtrs Y, int64_t ldy, float* c_saved,
                         hipStream_t s) {
  FastArgs a{};
  // the backward-ordered coefficient copy goes to the caller's buffer, or to the plan's own
  // copy, which every backward that is not handed a saved copy rewrites first
  a.csave = c_saved ? c_saved : p->fast.coef_bwd;
  a.pos = p->fast.bwd_pos;
  a.nslot = p->fast.coef_slots;
  a.bpad = p->fast.bwd_pad;
  a.nbpad = p->fast.nbpad;
  a.slots = p->fast.bwd_slots;
  a.frag = p->fout->dev.fs16;
  a.T = T;
  a.nblk_in = p->fin->dev.nblk;
  a.nblk_out = p->fout->dev.nblk;
  a.X = X.one;
  a.Xs = X.many;
  a.ldx = (long)ldx;
  a.Y = const_cast<void*>(Y.one);
  a.Ys = const_cast<void* const*>(Y.many);
  a.ldy = (long)ldy;
  a.c = c;
  a.cs = cs;
  a.scale = scale;
  a.beta = beta;
  const dim3 grid((unsigned)((T + kTT - 1) / kTT), (unsigned)count);
  const size_t lds = fast128_lds_bytes(a.nblk_in);
  hipEvent_t e0, e1;
  take_timing_events(&e0, &e1);
  if (T == 0) {   // no tiles: the copy alone
    if (!c_saved) return hipSuccess;
    const dim3 g((unsigned)((a.nslot + a.nbpad + 255) / 256), (unsigned)count);
    hipLaunchKernelGGL(scatter_bwd_coef, g, dim3(256), 0, s, c, cs, a.pos, a.nslot, a.bpad, a.nbpad, a.slots + 256,
                       c_saved);
    return hipGetLastError();
  }
  rec(e0, s);
  if (beta != 0.f)
    hipLaunchKernelGGL((fwd128<true, false>), grid, dim3(kThreads), lds, s, a, p->fast.fwd_pl, p->fast.fwd_st,
                       p->fast.fwd_em);
  else
    hipLaunchKernelGGL((fwd128<false, false>), grid, dim3(kThreads), lds, s, a, p->fast.fwd_pl, p->fast.fwd_st,
                       p->fast.fwd_em);
  rec(e1, s);
  return hipGetLastError();
}

// Floats of backward scratch (the backward-ordered coefficient copy, then the dC partial rows of
// every tile) that a single-adapter call of T tokens uses; the partial rows start 256-byte aligned.
size_t fast128_bwd_scratch_floats(const ff_plan* p, int T, size_t* partial_off) {
  const int tt = p->fast.bwd16 ? kTT16 : kTT;
  const size_t pstride = fast128_partial_floats((size_t)p->fast.bwd_slots);
  const size_t off = (pstride + 63) / 64 * 64;
  if (partial_off) *partial_off = off;
  return off + (size_t)((T + tt - 1) / tt) * pstride;
}

hipError_t launch_bwd128(const ff_plan* p, int count, int T, ActPtrs X, int64_t ldx, ActPtrs G, int64_t ldg,
                         const float* c, const float* const* cs, float scale, float beta_dx, ActPtrs dX,
                         int64_t lddx, bool want_dx, int accumulate_dc, float* dC, float* const* dCs, bool want_dc,
                         const float* c_saved, hipStream_t s, const BwdScratch* ws) {
  if (ws && count != 1) return hipErrorInvalidValue;   // a caller's scratch serves one adapter
  FastArgs a{};
  a.frag = p->fin->dev.fs16;
  a.T = T;
  a.nblk_in = p->fin->dev.nblk;
  a.nblk_out = p->fout->dev.nblk;
  a.X = X.one;
  a.Xs = X.many;
  a.ldx = (long)ldx;
  a.G = G.one;
  a.Gs = G.many;
  a.ldg = (long)ldg;
  a.Y = const_cast<void*>(dX.one);
  a.Ys = const_cast<void* const*>(dX.many);
  a.ldy = (long)lddx;
  a.c = c;
  a.cs = cs;
  a.scale = scale;
  a.beta = beta_dx;
  a.slots = p->fast.bwd_slots;
  a.pstride = (int)fast128_partial_floats((size_t)a.slots);
  a.partial = p->partial;
  float* copy = p->fast.coef_bwd;   // where the coefficients are put in backward slot order
  if (ws) {   // the caller's scratch instead of the plan's workspace
    size_t off = 0;
    if (fast128_bwd_scratch_floats(p, T, &off) > ws->floats) return hipErrorInvalidValue;
    copy = ws->base;
    a.partial = ws->base + off;
  }
  a.cb = c_saved ? c_saved : copy;
  const bool b16 = p->fast.bwd16 != 0;
  const int tt = b16 ? kTT16 : kTT;
  const long ntiles = (T + tt - 1) / tt;
  a.ntiles = ntiles;
  hipEvent_t e0, e1;
  take_timing_events(&e0, &e1);
  if (T > 0 && want_dx && !c_saved) {
    const int nslot = p->fast.coef_slots;
    if (ws) {   // the plan's copy was cleared once at creation; a shared scratch holds anything
      const int n = a.slots + 256;
      hipLaunchKernelGGL(fill_zero, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, copy, n);
    }
    const dim3 g((unsigned)((nslot + p->fast.nbpad + 255) / 256), (unsigned)count);
    hipLaunchKernelGGL(scatter_bwd_coef, g, dim3(256), 0, s, c, cs, p->fast.bwd_pos, nslot, p->fast.bwd_pad,
                       p->fast.nbpad, a.slots + 256, copy);
  }
  if (T > 0 && (want_dx || want_dc)) {
    const dim3 grid((unsigned)ntiles, (unsigned)count);
    const int4* pl = p->fast.bwd_pl;
    const unsigned* st = p->fast.bwd_st;
    const unsigned* em = p->fast.bwd_em;
    const bool beta = beta_dx != 0.f;
    rec(e0, s);
    if (b16) {
      const size_t lds = fast16_lds_bytes(a.nblk_out);
      const dim3 blk(kThreads16);
      if (want_dx && want_dc && beta)
        hipLaunchKernelGGL((bwd16<true, true, true, false>), grid, blk, lds, s, a, pl, st);
      else if (want_dx && want_dc)
        hipLaunchKernelGGL((bwd16<true, true, false, false>), grid, blk, lds, s, a, pl, st);
      else if (want_dx && beta)
        hipLaunchKernelGGL((bwd16<true, false, true, false>), grid, blk, lds, s, a, pl, st);
      else if (want_dx)
        hipLaunchKernelGGL((bwd16<true, false, false, false>), grid, blk, lds, s, a, pl, st);
      else
        hipLaunchKernelGGL((bwd16<false, true, false, false>), grid, blk, lds, s, a, pl, st);
    } else {
    const size_t lds = fast128_lds_bytes(a.nblk_out);
    if (want_dx && want_dc && beta)
      hipLaunchKernelGGL((bwd128<true, true, true, false>), grid, dim3(kThreads), lds, s, a, pl, st, em);
    else if (want_dx && want_dc)
      hipLaunchKernelGGL((bwd128<true, true, false, false>), grid, dim3(kThreads), lds, s, a, pl, st, em);
    else if (want_dx && beta)
      hipLaunchKernelGGL((bwd128<true, false, true, false>), grid, dim3(kThreads), lds, s, a, pl, st, em);
    else if (want_dx)
      hipLaunchKernelGGL((bwd128<true, false, false, false>), grid, dim3(kThreads), lds, s, a, pl, st, em);
    else
      hipLaunchKernelGGL((bwd128<false, true, false, false>), grid, dim3(kThreads), lds, s, a, pl, st, em);
    }
    rec(e1, s);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (want_dc) {
    const int nred = (a.slots + 63) / 64;
    const int npad = accumulate_dc ? 0 : p->fast.npad;
    const int nzero = (npad + 64 * kRedWaves - 1) / (64 * kRedWaves);
    if (nred + nzero > 0) {
      const dim3 grid((unsigned)(nred + nzero), (unsigned)count);
      hipLaunchKernelGGL(reduce128, grid, dim3(64 * kRedWaves), 0, s, a.partial, ntiles, a.slots, a.pstride,
                         p->fast.bwd_dst, scale, accumulate_dc, dC, dCs, p->fast.pad, npad, nred);
    }
  }
  return hipGetLastError();
}


hipError_t launch_fwd128_group(const ff_plan_group* g, int T, const int* tokens, const void* const* X, int64_t ldx,
                               const float* const* cs, float scale, float beta, void* const* Y, int64_t ldy,
                               hipStream_t s) {
  const ff_plan* p = g->ref;
  FastArgs a{};
  a.frag = p->fout->dev.fs16;
  a.T = T;
  a.nblk_in = p->fin->dev.nblk;
  a.nblk_out = p->fout->dev.nblk;
  a.Xs = X;
  a.ldx = (long)ldx;
  a.Ys = Y;
  a.ldy = (long)ldy;
  a.cs = cs;
  a.scale = scale;
  a.beta = beta;
  a.group = g->fast;
  a.tokens = tokens;
  const dim3 grid((unsigned)((T + kTT - 1) / kTT), (unsigned)g->count);
  const size_t lds = fast128_lds_bytes(a.nblk_in);
  hipEvent_t e0, e1;
  take_timing_events(&e0, &e1);
  rec(e0, s);
  if (beta != 0.f)
    hipLaunchKernelGGL((fwd128<true, true>), grid, dim3(kThreads), lds, s, a, nullptr, nullptr, nullptr);
  else
    hipLaunchKernelGGL((fwd128<false, true>), grid, dim3(kThreads), lds, s, a, nullptr, nullptr, nullptr);
  rec(e1, s);
  return hipGetLastError();
}

hipError_t launch_bwd128_group(const ff_plan_group* g, int T, const int* tokens, const void* const* X, int64_t ldx,
                               const void* const* G, int64_t ldg, const float* const* cs, float scale, float beta_dx,
                               void* const* dX, int64_t lddx, bool want_dx, int accumulate_dc, float* const* dCs,
                               bool want_dc, hipStream_t s) {
  const ff_plan* p = g->ref;
  const unsigned count = (unsigned)g->count;
  FastArgs a{};
  a.frag = p->fin->dev.fs16;
  a.T = T;
  a.nblk_in = p->fin->dev.nblk;
  a.nblk_out = p->fout->dev.nblk;
  a.Xs = X;
  a.ldx = (long)ldx;
  a.Gs = G;
  a.ldg = (long)ldg;
  a.Ys = dX;
  a.ldy = (long)lddx;
  a.cs = cs;
  a.scale = scale;
  a.beta = beta_dx;
  a.group = g->fast;
  a.tokens = tokens;
  hipEvent_t e0, e1;
  take_timing_events(&e0, &e1);
  if (want_dx && T > 0) {   // every adapter's coefficients in its backward's slot order
    const int nc = g->max_fast_slots + 256;
    hipLaunchKernelGGL(clear_copy_group, dim3((unsigned)((nc + 255) / 256), count), dim3(256), 0, s, g->fast);
    hipLaunchKernelGGL(scatter_bwd_coef_group, dim3((unsigned)((g->max_fast_items + 255) / 256), count), dim3(256),
                       0, s, cs, g->fast);
  }
  const bool beta = beta_dx != 0.f;
  rec(e0, s);
  // adapters whose plans run 16-token tiles, then those that run 8-token tiles: each kernel skips
  // the other kind (no tiles at all for T = 0: the reduction below writes zeros)
  if (T > 0 && g->fast16) {
    const dim3 grid((unsigned)((T + kTT16 - 1) / kTT16), count);
    const size_t lds = fast16_lds_bytes(a.nblk_out);
    const dim3 blk(kThreads16);
    if (want_dx && want_dc && beta)
      hipLaunchKernelGGL((bwd16<true, true, true, true>), grid, blk, lds, s, a, nullptr, nullptr);
    else if (want_dx && want_dc)
      hipLaunchKernelGGL((bwd16<true, true, false, true>), grid, blk, lds, s, a, nullptr, nullptr);
    else if (want_dx && beta)
      hipLaunchKernelGGL((bwd16<true, false, true, true>), grid, blk, lds, s, a, nullptr, nullptr);
    else if (want_dx)
      hipLaunchKernelGGL((bwd16<true, false, false, true>), grid, blk, lds, s, a, nullptr, nullptr);
    else
      hipLaunchKernelGGL((bwd16<false, true, false, true>), grid, blk, lds, s, a, nullptr, nullptr);
  }
  if (T > 0 && g->fast8) {
    const dim3 grid((unsigned)((T + kTT - 1) / kTT), count);
    const size_t lds = fast128_lds_bytes(a.nblk_out);
    const dim3 blk(kThreads);
    if (want_dx && want_dc && beta)
      hipLaunchKernelGGL((bwd128<true, true, true, true>), grid, blk, lds, s, a, nullptr, nullptr, nullptr);
    else if (want_dx && want_dc)
      hipLaunchKernelGGL((bwd128<true, true, false, true>), grid, blk, lds, s, a, nullptr, nullptr, nullptr);
    else if (want_dx && beta)
      hipLaunchKernelGGL((bwd128<true, false, true, true>), grid, blk, lds, s, a, nullptr, nullptr, nullptr);
    else if (want_dx)
      hipLaunchKernelGGL((bwd128<true, false, false, true>), grid, blk, lds, s, a, nullptr, nullptr, nullptr);
    else
      hipLaunchKernelGGL((bwd128<false, true, false, true>), grid, blk, lds, s, a, nullptr, nullptr, nullptr);
  }
  rec(e1, s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (want_dc) {
    const int nred = (g->max_fast_slots + 63) / 64;
    const int nzero = accumulate_dc ? 0 : (g->max_fast_npad + 64 * kRedWaves - 1) / (64 * kRedWaves);
    hipLaunchKernelGGL(reduce128_group, dim3((unsigned)(nred + nzero), count), dim3(64 * kRedWaves), 0, s, g->fast,
                       tokens, T, scale, accumulate_dc, dCs);
  }
  return hipGetLastError();
}

}  // namespace ff
