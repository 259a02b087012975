// Fused forward / backward for frames whose diagonal block is 128 x 128
// (k = 64, e.g. every 4096-wide Llama projection with rho = 64), bf16
// activations.
//
// Layout.  A workgroup owns a tile of 8 tokens.  The coefficients of one side
// (z = P_in^T x forward, u = P_out^T g backward) live in LDS coefficient-major:
// row c holds the 8 tokens' bf16 values (16 bytes), so every sparse access of
// C's random support is one 16-byte LDS read covering the whole tile.  Rows are
// XOR-swizzled inside each 128-row block so that the MFMA-side reads and writes
// (8 consecutive coefficients of one token, four tokens' lanes per row) hit
// distinct banks.
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
// of C for v = C z, whole columns for q = C^T u), and the coefficient vector is
// in the plan's order, which is the forward stream's order: forward slots read
// their coefficients with coalesced loads that do not wait for the entries.
// The next pair's stream chunk is loaded while the current pair is synthesised.
// The backward runs one stream per input pair twice: first for this tile's
// share of dC_e = sum_t u_t[a_e] z_t[b_e] (v_dot2_f32_bf16 over token pairs),
// then for q = C^T u; partial dC sums go to a workspace reduced in a fixed
// order by a second kernel.
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
constexpr int kCh = 16;   // stream slots per lane held in registers at once

constexpr unsigned kValid = 1u << 25, kEnd = 1u << 24;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16;

__device__ __forceinline__ int swz(int blk, int o) { return o ^ ((o >> 2) & 4) ^ ((blk & 1) << 1); }

__device__ __forceinline__ float lo_bf(unsigned w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf(unsigned w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ unsigned pack_bf2(float a, float b) {
  bf16x2 p = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(unsigned, p);
}

__device__ __forceinline__ u16 to_bf(float a) { return __builtin_bit_cast(u16, (__bf16)a); }

// Ordering point between phases that hand data through a wave's private LDS tile:
// LDS instructions of one wave execute in order, so only the compiler must not move
// accesses across it.
__device__ __forceinline__ void wave_lds_fence() { __asm__ volatile("" ::: "memory"); }

struct Frag {
  bf16x8 f[kHT][kKT];
};

// Stage the 16 KB of upper-half synthesis fragments through LDS (once per workgroup) and load
// this wave's copy.  `stage` must be free LDS of that size; it may be reused after return.
// The fragment array is ordered [row tile][contraction step][lane], so the upper half is its
// first half.
__device__ __forceinline__ void load_frag(const void* fs16, u32x4* stage, int lane, Frag& F) {
  const u32x4* src = reinterpret_cast<const u32x4*>(fs16);
  for (int i = threadIdx.x; i < kHT * kKT * 64; i += kThreads) stage[i] = src[i];
  __syncthreads();
#pragma unroll
  for (int mt = 0; mt < kHT; ++mt)
#pragma unroll
    for (int ks = 0; ks < kKT; ++ks) F.f[mt][ks] = __builtin_bit_cast(bf16x8, stage[(mt * kKT + ks) * 64 + lane]);
  __syncthreads();
}

// acc[mt] = sum_ks B[mt][ks] * b[ks] for the 8 row tiles of the block; rows 64..127 use the
// upper-half fragments on the input with its odd complex components negated.  With flip
// (analysis) odd real inputs are negated first.  A lane's 8 inputs of a contraction step are
// real indices 32 ks + 8 q + j: odd j is the high half of each word, odd complex index is
// words 1 and 3.
__device__ __forceinline__ void mfma_block(const Frag& F, const u32x4 (&b)[kKT], f32x4 (&acc)[kMT], bool flip) {
  const unsigned d = flip ? 0x80000000u : 0u;
  const u32x4 m_top = {d, d, d, d};
  const u32x4 m_bot = {d, d ^ 0x80008000u, d, d ^ 0x80008000u};
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < kKT; ++ks) {
    const bf16x8 bt = __builtin_bit_cast(bf16x8, b[ks] ^ m_top);
    const bf16x8 bb = __builtin_bit_cast(bf16x8, b[ks] ^ m_bot);
#pragma unroll
    for (int mt = 0; mt < kHT; ++mt) {
      acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(F.f[mt][ks], bt, acc[mt], 0, 0, 0);
      acc[mt + kHT] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(F.f[mt][ks], bb, acc[mt + kHT], 0, 0, 0);
    }
  }
}

// Activation fragments of one column group: lane (token t, block bs of the pair, quarter q)
// reads 8 consecutive inputs per contraction step from a row-major token matrix.  The loads
// are unconditional (tokens past the tile's end re-read its last token) and nothing touches
// the registers until mfma_block, so they stay in flight; store_coef zeroes those columns and
// store_act skips them.
__device__ __forceinline__ void load_act(const u16* rows, long ld, int nt, int blk0, int lane, u32x4 (&b)[kKT]) {
  const int n = lane & 15, t = min(n & 7, nt - 1), bs = n >> 3, q = lane >> 4;
  const u16* p = rows + (long)t * ld + (blk0 + bs) * kW + 8 * q;
#pragma unroll
  for (int ks = 0; ks < kKT; ++ks) b[ks] = *reinterpret_cast<const u32x4*>(p + 32 * ks);
}

// Write an analysis result (odd outputs negated) into a coefficient-major LDS array whose
// block `blk0 + bs` starts at row (blk0 + bs - row_blk0) * 128.  Columns of tokens past the
// tile's end are written as zeros.
__device__ __forceinline__ void store_coef(u16* lds, int blk0, int row_blk0, int nt, int lane,
                                           const f32x4 (&acc)[kMT]) {
  const int n = lane & 15, t = n & 7, bs = n >> 3, q = lane >> 4;
  const int blk = blk0 + bs;
  const float keep = t < nt ? 1.f : 0.f;
  u16* base = lds + (long)(blk - row_blk0) * kW * kTT + t;
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int o = 16 * mt + 4 * q + j;
      const float v = (j & 1) ? -keep * acc[mt][j] : keep * acc[mt][j];
      base[swz(blk, o) * kTT] = to_bf(v);
    }
}

// Gather the synthesis operand of the pair tile (rows bs*128 + swz(bs, o), 8 tokens per row).
__device__ __forceinline__ void load_tile_act(const u16* tile, int lane, u32x4 (&b)[kKT]) {
  const int n = lane & 15, t = n & 7, bs = n >> 3, q = lane >> 4;
  const u16* base = tile + bs * kW * kTT + t;
#pragma unroll
  for (int ks = 0; ks < kKT; ++ks) {
    unsigned w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int o = 32 * ks + 8 * q + 2 * i;
      const unsigned e0 = base[swz(bs, o) * kTT], e1 = base[swz(bs, o + 1) * kTT];
      w[i] = e0 | (e1 << 16);
    }
    b[ks] = u32x4{w[0], w[1], w[2], w[3]};
  }
}

// y[t][(blk0+bs)*128 + o] = scale * acc (+ beta * y)
__device__ __forceinline__ void store_act(u16* rows, long ld, int nt, int blk0, int lane, const f32x4 (&acc)[kMT],
                                          float scale, float beta) {
  const int n = lane & 15, t = n & 7, bs = n >> 3, q = lane >> 4;
  if (t >= nt) return;
  u16* p = rows + (long)t * ld + (blk0 + bs) * kW + 4 * q;
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt) {
    f32x4 r = acc[mt] * scale;
    uint2* dst = reinterpret_cast<uint2*>(p + 16 * mt);
    if (beta != 0.f) {
      const uint2 old = *dst;
      r[0] += beta * lo_bf(old.x);
      r[1] += beta * hi_bf(old.x);
      r[2] += beta * lo_bf(old.y);
      r[3] += beta * hi_bf(old.y);
    }
    *dst = make_uint2(pack_bf2(r[0], r[1]), pack_bf2(r[2], r[3]));
  }
}

__device__ __forceinline__ void zero_tile(u16* tile, int lane) {
  u32x4* tz = reinterpret_cast<u32x4*>(tile);
  wave_lds_fence();
#pragma unroll
  for (int i = 0; i < 4; ++i) tz[lane + 64 * i] = u32x4{0u, 0u, 0u, 0u};
  wave_lds_fence();
}

// a[0..7] += c * (8 bf16 tokens of source row); at the end of a row, write it to the tile.
__device__ __forceinline__ void accum_row(unsigned e, float c, const u16* src, u16* tile, float (&a)[8]) {
  const u32x4 zv = *reinterpret_cast<const u32x4*>(src + (e & 0xffffu) * kTT);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const unsigned w = zv[j];
    a[2 * j] = fmaf(c, lo_bf(w), a[2 * j]);
    a[2 * j + 1] = fmaf(c, hi_bf(w), a[2 * j + 1]);
  }
  if (e & kEnd) {
    reinterpret_cast<u32x4*>(tile)[(e >> 16) & 0xffu] =
        u32x4{pack_bf2(a[0], a[1]), pack_bf2(a[2], a[3]), pack_bf2(a[4], a[5]), pack_bf2(a[6], a[7])};
#pragma unroll
    for (int j = 0; j < 8; ++j) a[j] = 0.f;
  }
}

// ---------------------------------------------------------------- forward stream chunks

struct FwdChunk {
  unsigned en[kCh];
  float cc[kCh];
};

// Load slots k0 .. k0+kCh-1 of a forward stream: entries and their coefficients, which sit at
// plan index rowinfo.x + lane; loads are clamped to real rows/lanes and masked when used.
__device__ __forceinline__ void fwd_load(const unsigned* __restrict__ st, const int2* __restrict__ ri, int off,
                                         int len, int k0, const float* __restrict__ cv, int lane, FwdChunk& ch) {
#pragma unroll
  for (int i = 0; i < kCh; ++i) {
    const int r = off + min(k0 + i, len - 1);
    const int2 info = ri[r];
    ch.en[i] = st[(long)r * 64 + lane];
    ch.cc[i] = cv[info.x + min(lane, info.y - 1)];
  }
}

__device__ __forceinline__ void fwd_compute(const FwdChunk& ch, int len, int k0, const u16* zL, u16* tile,
                                            float (&a)[8]) {
#pragma unroll
  for (int i = 0; i < kCh; ++i) {
    if (k0 + i < len) {   // uniform
      const unsigned e = ch.en[i];
      accum_row(e, (e & kValid) ? ch.cc[i] : 0.f, zL, tile, a);
    }
  }
}

// ---------------------------------------------------------------- backward stream chunks

struct BwdChunk {
  uint2 en[kCh];
  float cc[kCh];
};

__device__ __forceinline__ void bwd_load_entries(const uint2* __restrict__ st, int len, int k0, int lane,
                                                 BwdChunk& ch) {
#pragma unroll
  for (int i = 0; i < kCh; ++i) ch.en[i] = st[(long)min(k0 + i, len - 1) * 64 + lane];
}

// Coefficients of the loaded entries (empty slots read entry 0 and are masked when used).
__device__ __forceinline__ void bwd_load_coeffs(const float* __restrict__ cv, BwdChunk& ch) {
#pragma unroll
  for (int i = 0; i < kCh; ++i) ch.cc[i] = cv[ch.en[i].y];
}

// This tile's share of dC / s for the chunk's slots, written to part (one float per slot).
__device__ __forceinline__ void bwd_sddmm(const BwdChunk& ch, int len, int k0, const u16* uL, const u16* tile,
                                          float* __restrict__ part, int lane) {
#pragma unroll
  for (int i = 0; i < kCh; ++i) {
    if (k0 + i < len) {   // uniform
      const unsigned e = ch.en[i].x;
      const u32x4 uv = *reinterpret_cast<const u32x4*>(uL + (e & 0xffffu) * kTT);
      const u32x4 zv = *reinterpret_cast<const u32x4*>(tile + ((e >> 16) & 0xffu) * kTT);
      float s = 0.f;
  #pragma unroll
      for (int j = 0; j < 4; ++j) {
        // copy the elements out first: bit-casting a vector element expression directly reads
        // element 0 with this compiler
        const unsigned uw = uv[j], zw = zv[j];
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, uw), __builtin_bit_cast(bf16x2, zw), s, false);
      }
      part[(long)(k0 + i) * 64 + lane] = (e & kValid) ? s : 0.f;
    }
  }
}

__device__ __forceinline__ void bwd_spmm(const BwdChunk& ch, int len, int k0, const u16* uL, u16* tile,
                                         float (&a)[8]) {
#pragma unroll
  for (int i = 0; i < kCh; ++i) {
    if (k0 + i < len) {   // uniform
      const unsigned e = ch.en[i].x;
      accum_row(e, (e & kValid) ? ch.cc[i] : 0.f, uL, tile, a);
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
  float scale, beta;
  int want_dx, want_dc;
  const int* off;     // per pair: first stream row
  const int* len;     // per pair: stream rows
  const unsigned* fst;
  const int2* fri;
  const uint2* bst;
  int slots;          // dC partials per tile
  float* partial;     // [batch][tile][slots]
  long ntiles;
};

// Analysis of every pair of blocks of a tile into a coefficient-major LDS array, two pairs'
// inputs in flight per wave.
__device__ __forceinline__ void analysis_phase(const Frag& F, const u16* rows, long ld, int nt, int np, int wave,
                                               int lane, u16* lds) {
  u32x4 bA[kKT], bB[kKT];
  if (wave < np) load_act(rows, ld, nt, 2 * wave, lane, bA);
  if (wave + kWaves < np) load_act(rows, ld, nt, 2 * (wave + kWaves), lane, bB);
  for (int p = wave; p < np; p += 2 * kWaves) {
    {
      f32x4 acc[kMT];
      mfma_block(F, bA, acc, true);
      store_coef(lds, 2 * p, 0, nt, lane, acc);
    }
    if (p + 2 * kWaves < np) load_act(rows, ld, nt, 2 * (p + 2 * kWaves), lane, bA);
    if (p + kWaves < np) {
      f32x4 acc[kMT];
      mfma_block(F, bB, acc, true);
      store_coef(lds, 2 * (p + kWaves), 0, nt, lane, acc);
      if (p + 3 * kWaves < np) load_act(rows, ld, nt, 2 * (p + 3 * kWaves), lane, bB);
    }
  }
}

__global__ void __launch_bounds__(kThreads, 2) fwd128(FastArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  u16* zL = reinterpret_cast<u16*>(smem);                          // n rows x 8 tokens
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  u16* tile = zL + (long)a.nblk_in * kW * kTT + wave * (2 * kW * kTT);
  const int bi = blockIdx.y;
  const int t0 = blockIdx.x * kTT, nt = min(kTT, a.T - t0);
  const u16* X = reinterpret_cast<const u16*>(a.Xs ? a.Xs[bi] : a.X) + (long)t0 * a.ldx;
  u16* Y = reinterpret_cast<u16*>(a.Ys ? a.Ys[bi] : a.Y) + (long)t0 * a.ldy;
  const float* cv = a.cs ? a.cs[bi] : a.c;
  const int npo = a.nblk_out / 2;

  // first stream chunk of this wave's first output pair, in flight during the analysis
  FwdChunk ch;
  if (wave < npo && a.len[wave] > 0) fwd_load(a.fst, a.fri, a.off[wave], a.len[wave], 0, cv, lane, ch);

  Frag F;
  load_frag(a.frag, reinterpret_cast<u32x4*>(smem), lane, F);
  analysis_phase(F, X, a.ldx, nt, a.nblk_in / 2, wave, lane, zL);
  __syncthreads();

  for (int p = wave; p < npo; p += kWaves) {
    // v = C z for this pair into the tile
    const int off = a.off[p], len = a.len[p];
    zero_tile(tile, lane);
    float acc8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < len; k0 += kCh) {
      if (k0 > 0) fwd_load(a.fst, a.fri, off, len, k0, cv, lane, ch);
      fwd_compute(ch, len, k0, zL, tile, acc8);
    }
    wave_lds_fence();
    // next pair's first chunk flies during this pair's synthesis
    const int pn = p + kWaves;
    if (pn < npo && a.len[pn] > 0) fwd_load(a.fst, a.fri, a.off[pn], a.len[pn], 0, cv, lane, ch);
    // y = beta y + s P_out v
    u32x4 b[kKT];
    f32x4 acc[kMT];
    load_tile_act(tile, lane, b);
    wave_lds_fence();
    mfma_block(F, b, acc, false);
    store_act(Y, a.ldy, nt, 2 * p, lane, acc, a.scale, a.beta);
  }
}

__global__ void __launch_bounds__(kThreads, 2) bwd128(FastArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  u16* uL = reinterpret_cast<u16*>(smem);                          // m rows x 8 tokens
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  u16* tile = uL + (long)a.nblk_out * kW * kTT + wave * (2 * kW * kTT);
  const int bi = blockIdx.y;
  const int t0 = blockIdx.x * kTT, nt = min(kTT, a.T - t0);
  const u16* G = reinterpret_cast<const u16*>(a.Gs ? a.Gs[bi] : a.G) + (long)t0 * a.ldg;
  const u16* X = a.want_dc ? reinterpret_cast<const u16*>(a.Xs ? a.Xs[bi] : a.X) + (long)t0 * a.ldx : nullptr;
  u16* dX = a.want_dx ? reinterpret_cast<u16*>(a.Ys ? a.Ys[bi] : a.Y) + (long)t0 * a.ldy : nullptr;
  const float* cv = a.cs ? a.cs[bi] : a.c;
  float* part = a.partial + ((long)bi * a.ntiles + blockIdx.x) * a.slots;
  const int npi = a.nblk_in / 2;

  // this wave's first input pair: stream entries and x in flight during the analysis of g
  BwdChunk ch;
  u32x4 bx[kKT];
  if (wave < npi) {
    if (a.len[wave] > 0) bwd_load_entries(a.bst + (long)a.off[wave] * 64, a.len[wave], 0, lane, ch);
    if (a.want_dc) load_act(X, a.ldx, nt, 2 * wave, lane, bx);
  }

  Frag F;
  load_frag(a.frag, reinterpret_cast<u32x4*>(smem), lane, F);
  analysis_phase(F, G, a.ldg, nt, a.nblk_out / 2, wave, lane, uL);
  __syncthreads();

  for (int p = wave; p < npi; p += kWaves) {
    const int len = a.len[p];
    const uint2* st = a.bst + (long)a.off[p] * 64;
    if (a.want_dx && len > 0) bwd_load_coeffs(cv, ch);
    if (a.want_dc) {
      // z = P_in^T x for this pair, then this tile's share of dC
      f32x4 acc[kMT];
      mfma_block(F, bx, acc, true);
      store_coef(tile, 2 * p, 2 * p, nt, lane, acc);
      wave_lds_fence();
      if (p + kWaves < npi) load_act(X, a.ldx, nt, 2 * (p + kWaves), lane, bx);
      float* pp = part + (long)a.off[p] * 64;
      for (int k0 = 0; k0 < len; k0 += kCh) {
        if (k0 > 0) bwd_load_entries(st, len, k0, lane, ch);
        bwd_sddmm(ch, len, k0, uL, tile, pp, lane);
      }
      wave_lds_fence();
      if (a.want_dx && len > kCh) {   // the stream is reread for q
        bwd_load_entries(st, len, 0, lane, ch);
        bwd_load_coeffs(cv, ch);
      }
    }
    if (a.want_dx) {
      // q = C^T u for this pair, then dX = beta dX + s P_in q
      zero_tile(tile, lane);
      float acc8[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      for (int k0 = 0; k0 < len; k0 += kCh) {
        if (k0 > 0) {
          bwd_load_entries(st, len, k0, lane, ch);
          bwd_load_coeffs(cv, ch);
        }
        bwd_spmm(ch, len, k0, uL, tile, acc8);
      }
      wave_lds_fence();
    }
    const int pn = p + kWaves;
    if (pn < npi && a.len[pn] > 0) bwd_load_entries(a.bst + (long)a.off[pn] * 64, a.len[pn], 0, lane, ch);
    if (a.want_dx) {
      u32x4 b[kKT];
      f32x4 acc[kMT];
      load_tile_act(tile, lane, b);
      wave_lds_fence();
      mfma_block(F, b, acc, false);
      store_act(dX, a.ldy, nt, 2 * p, lane, acc, a.scale, a.beta);
    }
  }
}

// dC[j] = [dC[j] +] s * sum_tiles partial[tile][slot] for every valid slot of the backward
// streams (j = the slot's plan index).  Eight waves split the tiles; their sums are combined
// in a fixed order.
__global__ void __launch_bounds__(512) reduce128(const float* __restrict__ partial, long ntiles, int slots,
                                                 const uint2* __restrict__ bst, float scale, int accumulate,
                                                 float* dC, float* const* dCs) {
  __shared__ float red[8][64];
  const int bi = blockIdx.y;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int slot = blockIdx.x * 64 + lane;
  float s = 0.f;
  if (slot < slots) {
    const float* p = partial + (long)bi * ntiles * slots + slot;
    float s1 = 0.f, s2 = 0.f, s3 = 0.f;
    long t = w;
    for (; t + 24 < ntiles; t += 32) {
      s += p[t * slots];
      s1 += p[(t + 8) * slots];
      s2 += p[(t + 16) * slots];
      s3 += p[(t + 24) * slots];
    }
    for (; t < ntiles; t += 8) s += p[t * slots];
    s = (s + s1) + (s2 + s3);
  }
  red[w][lane] = s;
  __syncthreads();
  if (w == 0 && slot < slots) {
    float tot = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) tot += red[i][lane];
    const uint2 en = bst[slot];
    if (en.x & kValid) {
      float* out = dCs ? dCs[bi] : dC;
      const float v = scale * tot;
      out[en.y] = accumulate ? out[en.y] + v : v;
    }
  }
}

void rec(hipEvent_t ev, hipStream_t s) {
  if (ev) (void)hipEventRecord(ev, s);
}

}  // namespace

hipError_t configure_fast128() {
  static hipError_t once = [] {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&fwd128),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLdsBytes);
    if (e == hipSuccess)
      e = hipFuncSetAttribute(reinterpret_cast<const void*>(&bwd128), hipFuncAttributeMaxDynamicSharedMemorySize,
                              kMaxLdsBytes);
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

hipError_t launch_fwd128(const ff_plan* p, int count, int T, ActPtrs X, int64_t ldx, const float* c,
                         const float* const* cs, float scale, float beta, ActPtrs Y, int64_t ldy, hipStream_t s) {
  FastArgs a{};
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
  a.off = p->fast.fwd_off;
  a.len = p->fast.fwd_len;
  a.fst = p->fast.fwd_st;
  a.fri = p->fast.fwd_ri;
  const dim3 grid((unsigned)((T + kTT - 1) / kTT), (unsigned)count);
  hipEvent_t e0, e1;
  take_timing_events(&e0, &e1);
  rec(e0, s);
  hipLaunchKernelGGL(fwd128, grid, dim3(kThreads), fast128_lds_bytes(a.nblk_in), s, a);
  rec(e1, s);
  return hipGetLastError();
}

hipError_t launch_bwd128(const ff_plan* p, int count, int T, ActPtrs X, int64_t ldx, ActPtrs G, int64_t ldg,
                         const float* c, const float* const* cs, float scale, float beta_dx, ActPtrs dX,
                         int64_t lddx, bool want_dx, int accumulate_dc, float* dC, float* const* dCs, bool want_dc,
                         hipStream_t s) {
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
  a.want_dx = want_dx;
  a.want_dc = want_dc;
  a.off = p->fast.bwd_off;
  a.len = p->fast.bwd_len;
  a.bst = p->fast.bwd_st;
  a.slots = p->fast.bwd_slots;
  a.partial = p->partial;
  const long ntiles = (T + kTT - 1) / kTT;
  a.ntiles = ntiles;
  hipEvent_t e0, e1;
  take_timing_events(&e0, &e1);
  if (T > 0 && (want_dx || want_dc)) {
    const dim3 grid((unsigned)ntiles, (unsigned)count);
    rec(e0, s);
    hipLaunchKernelGGL(bwd128, grid, dim3(kThreads), fast128_lds_bytes(a.nblk_out), s, a);
    rec(e1, s);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (want_dc) {
    const dim3 grid((unsigned)((a.slots + 63) / 64), (unsigned)count);
    hipLaunchKernelGGL(reduce128, grid, dim3(512), 0, s, p->partial, ntiles, a.slots, a.bst, scale, accumulate_dc, dC,
                       dCs);
  }
  return hipGetLastError();
}

}  // namespace ff
