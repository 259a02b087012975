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
// Frame products.  The block B (synthesis) is held in 128 VGPRs by every wave
// for the whole kernel.  Analysis needs B^T; for these frames B^T = D B D with
// D = diag(+1, -1, +1, ...) (the realified DFT is symmetric up to the sign of
// its sine terms), so analysis flips the sign of odd inputs and odd outputs and
// reuses the same fragments.  One v_mfma_f32_16x16x32_bf16 column group is 16
// (token, block) pairs: the tile's 8 tokens times a pair of adjacent blocks.
//
// Sparse products.  After the shared coefficient array is complete, each wave
// streams over its own block pairs with a private 4 KB LDS tile: it builds the
// pair's 256 coefficients of v = C z (forward) or q = C^T u (backward) from a
// load-balanced, lane-interleaved entry stream prepared by the plan (each lane
// owns whole rows; entries of a row are consecutive), then applies the frame
// block and writes the activations.  The backward also forms this tile's
// share of dC_e = sum_t u_t[a_e] z_t[b_e] with v_dot2_f32_bf16 over token pairs
// and stores it as a partial sum; a second kernel reduces partials in a fixed
// order.
#include "ff_internal.h"

namespace ff {
namespace {

constexpr int kW = 128;   // block width
constexpr int kTT = 8;    // tokens per tile
constexpr int kMT = 8;    // 16-row output tiles per block
constexpr int kKT = 4;    // 32-wide contraction steps per block
constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;

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
  bf16x8 f[kMT][kKT];
};

__device__ __forceinline__ void load_frag(const void* fs16, int lane, Frag& F) {
  const bf16x8* src = reinterpret_cast<const bf16x8*>(fs16);
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
    for (int ks = 0; ks < kKT; ++ks) F.f[mt][ks] = src[(mt * kKT + ks) * 64 + lane];
}

// acc[mt] = sum_ks F[mt][ks] * b[ks]
__device__ __forceinline__ void mfma_block(const Frag& F, const u32x4 (&b)[kKT], f32x4 (&acc)[kMT]) {
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int ks = 0; ks < kKT; ++ks) {
    const bf16x8 bk = __builtin_bit_cast(bf16x8, b[ks]);
#pragma unroll
    for (int mt = 0; mt < kMT; ++mt) acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(F.f[mt][ks], bk, acc[mt], 0, 0, 0);
  }
}

// Activation fragments of one column group: lane (token t, block bs of the pair, quarter q)
// reads 8 consecutive inputs per contraction step from a row-major token matrix.
__device__ __forceinline__ void load_act(const u16* rows, long ld, int nt, int blk0, int lane, bool flip,
                                         u32x4 (&b)[kKT]) {
  const int n = lane & 15, t = n & 7, bs = n >> 3, q = lane >> 4;
  if (t < nt) {
    const u16* p = rows + (long)t * ld + (blk0 + bs) * kW + 8 * q;
#pragma unroll
    for (int ks = 0; ks < kKT; ++ks) b[ks] = *reinterpret_cast<const u32x4*>(p + 32 * ks);
    if (flip) {
#pragma unroll
      for (int ks = 0; ks < kKT; ++ks) b[ks] ^= 0x80000000u;   // negate odd coordinates
    }
  } else {
#pragma unroll
    for (int ks = 0; ks < kKT; ++ks) b[ks] = u32x4{0u, 0u, 0u, 0u};
  }
}

// Write an analysis result (odd outputs negated) into a coefficient-major LDS array whose
// block `blk0 + bs` starts at row (blk0 + bs - row_blk0) * 128.
__device__ __forceinline__ void store_coef(u16* lds, int blk0, int row_blk0, int lane, const f32x4 (&acc)[kMT]) {
  const int n = lane & 15, t = n & 7, bs = n >> 3, q = lane >> 4;
  const int blk = blk0 + bs;
  u16* base = lds + (long)(blk - row_blk0) * kW * kTT + t;
#pragma unroll
  for (int mt = 0; mt < kMT; ++mt)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int o = 16 * mt + 4 * q + j;
      const float v = (j & 1) ? -acc[mt][j] : acc[mt][j];
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

// v[row][t] = sum_{e in row} c_e * src[row_e][t] over a lane-interleaved stream; rows are written
// into `tile` when their last entry is seen.  The tile is zeroed first (rows without entries).
__device__ __forceinline__ void spmm_stream(const uint2* __restrict__ st, int len, const float* __restrict__ cv,
                                            const u16* src, u16* tile, int lane) {
  u32x4* tz = reinterpret_cast<u32x4*>(tile);
  wave_lds_fence();
#pragma unroll
  for (int i = 0; i < 4; ++i) tz[lane + 64 * i] = u32x4{0u, 0u, 0u, 0u};
  wave_lds_fence();
  float a[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int k = 0; k < len; ++k) {
    const uint2 en = st[(long)k * 64 + lane];
    if (en.x & kValid) {
      const float c = cv[en.y];
      const u32x4 zv = *reinterpret_cast<const u32x4*>(src + (en.x & 0xffffu) * kTT);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[2 * i] = fmaf(c, lo_bf(zv[i]), a[2 * i]);
        a[2 * i + 1] = fmaf(c, hi_bf(zv[i]), a[2 * i + 1]);
      }
      if (en.x & kEnd) {
        tz[(en.x >> 16) & 0xffu] = u32x4{pack_bf2(a[0], a[1]), pack_bf2(a[2], a[3]), pack_bf2(a[4], a[5]),
                                          pack_bf2(a[6], a[7])};
#pragma unroll
        for (int i = 0; i < 8; ++i) a[i] = 0.f;
      }
    }
  }
  wave_lds_fence();
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
  const uint2* st;
  const int* soff;    // dC streams (backward)
  const int* slen;
  const uint2* sst;
  int slots;          // dC slots per tile
  float* partial;     // [batch][tile][slots]
  long ntiles;
};

__global__ void __launch_bounds__(kThreads, 2) fwd128(FastArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  u16* zL = reinterpret_cast<u16*>(smem);                          // n rows x 8 tokens
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  u16* tile = zL + (long)a.nblk_in * kW * kTT + wave * (2 * kW * kTT);
  const int bi = blockIdx.y;
  const int t0 = blockIdx.x * kTT, nt = min(kTT, a.T - t0);
  const u16* X = reinterpret_cast<const u16*>(a.Xs ? a.Xs[bi] : a.X) + (long)t0 * a.ldx;
  u16* Y = reinterpret_cast<u16*>(a.Ys ? a.Ys[bi] : a.Y) + (long)t0 * a.ldy;
  const float* cv = a.cs ? a.cs[bi] : a.c;

  Frag F;
  load_frag(a.frag, lane, F);
  // z = P_in^T x for the tile, one pair of blocks per step
  for (int p = wave; p < a.nblk_in / 2; p += kWaves) {
    u32x4 b[kKT];
    f32x4 acc[kMT];
    load_act(X, a.ldx, nt, 2 * p, lane, true, b);
    mfma_block(F, b, acc);
    store_coef(zL, 2 * p, 0, lane, acc);
  }
  __syncthreads();
  // per output pair: v = C z into the wave's tile, then y = beta y + s P_out v
  for (int p = wave; p < a.nblk_out / 2; p += kWaves) {
    spmm_stream(a.st + (long)a.off[p] * 64, a.len[p], cv, zL, tile, lane);
    u32x4 b[kKT];
    f32x4 acc[kMT];
    load_tile_act(tile, lane, b);
    wave_lds_fence();
    mfma_block(F, b, acc);
    store_act(Y, a.ldy, nt, 2 * p, lane, acc, a.scale, a.beta);
  }
}

__global__ void __launch_bounds__(kThreads, 2) bwd128(FastArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  u16* uL = reinterpret_cast<u16*>(smem);                          // m rows x 8 tokens
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  u16* tile = uL + (long)a.nblk_out * kW * kTT + wave * (2 * kW * kTT);
  const int bi = blockIdx.y;
  const int t0 = blockIdx.x * kTT, nt = min(kTT, a.T - t0);
  const u16* G = reinterpret_cast<const u16*>(a.Gs ? a.Gs[bi] : a.G) + (long)t0 * a.ldg;
  const u16* X = a.want_dc ? reinterpret_cast<const u16*>(a.Xs ? a.Xs[bi] : a.X) + (long)t0 * a.ldx : nullptr;
  u16* dX = a.want_dx ? reinterpret_cast<u16*>(a.Ys ? a.Ys[bi] : a.Y) + (long)t0 * a.ldy : nullptr;
  const float* cv = a.cs ? a.cs[bi] : a.c;
  float* part = a.partial + ((long)bi * a.ntiles + blockIdx.x) * a.slots;

  Frag F;
  load_frag(a.frag, lane, F);
  // u = P_out^T g for the tile
  for (int p = wave; p < a.nblk_out / 2; p += kWaves) {
    u32x4 b[kKT];
    f32x4 acc[kMT];
    load_act(G, a.ldg, nt, 2 * p, lane, true, b);
    mfma_block(F, b, acc);
    store_coef(uL, 2 * p, 0, lane, acc);
  }
  __syncthreads();
  for (int p = wave; p < a.nblk_in / 2; p += kWaves) {
    if (a.want_dc) {
      // z = P_in^T x for this pair of input blocks, then this tile's share of dC
      u32x4 b[kKT];
      f32x4 acc[kMT];
      load_act(X, a.ldx, nt, 2 * p, lane, true, b);
      mfma_block(F, b, acc);
      store_coef(tile, 2 * p, 2 * p, lane, acc);
      wave_lds_fence();
      const uint2* st = a.sst + (long)a.soff[p] * 64;
      float* pp = part + (long)a.soff[p] * 64;
      for (int k = 0; k < a.slen[p]; ++k) {
        const uint2 en = st[(long)k * 64 + lane];
        float s = 0.f;
        if (en.x & kValid) {
          const u32x4 uv = *reinterpret_cast<const u32x4*>(uL + (en.x & 0xffffu) * kTT);
          const u32x4 zv = *reinterpret_cast<const u32x4*>(tile + ((en.x >> 16) & 0xffu) * kTT);
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            // copy the elements out first: bit-casting a vector element expression directly
            // reads element 0 with this compiler
            const unsigned uw = uv[i], zw = zv[i];
            s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, uw), __builtin_bit_cast(bf16x2, zw), s,
                                                false);
          }
        }
        pp[(long)k * 64 + lane] = s;
      }
      wave_lds_fence();
    }
    if (a.want_dx) {
      // q = C^T u for this pair, then dX = beta dX + s P_in q
      spmm_stream(a.st + (long)a.off[p] * 64, a.len[p], cv, uL, tile, lane);
      u32x4 b[kKT];
      f32x4 acc[kMT];
      load_tile_act(tile, lane, b);
      wave_lds_fence();
      mfma_block(F, b, acc);
      store_act(dX, a.ldy, nt, 2 * p, lane, acc, a.scale, a.beta);
    }
  }
}

// dC[e] = [dC[e] +] s * sum_tiles partial[tile][slot] for every valid slot of the dC streams.
// Eight waves split the tiles; their sums are combined in a fixed order.
__global__ void __launch_bounds__(512) reduce128(const float* __restrict__ partial, long ntiles, int slots,
                                                 const uint2* __restrict__ sst, float scale, int accumulate,
                                                 float* dC, float* const* dCs) {
  __shared__ float red[8][64];
  const int bi = blockIdx.y;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int slot = blockIdx.x * 64 + lane;
  float s = 0.f;
  if (slot < slots) {
    const float* p = partial + (long)bi * ntiles * slots + slot;
    for (long t = w; t < ntiles; t += 8) s += p[t * slots];
  }
  red[w][lane] = s;
  __syncthreads();
  if (w == 0 && slot < slots) {
    float tot = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) tot += red[i][lane];
    const uint2 en = sst[slot];
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

size_t fast128_lds_bytes(int nblk) { return (size_t)nblk * kW * kTT * 2 + (size_t)kWaves * 2 * kW * kTT * 2; }

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
  a.st = p->fast.fwd_st;
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
  a.st = p->fast.bwd_st;
  a.soff = p->fast.sdd_off;
  a.slen = p->fast.sdd_len;
  a.sst = p->fast.sdd_st;
  a.slots = p->fast.sdd_slots;
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
    hipLaunchKernelGGL(reduce128, grid, dim3(512), 0, s, p->partial, ntiles, a.slots, a.sst, scale, accumulate_dc, dC,
                       dCs);
  }
  return hipGetLastError();
}

}  // namespace ff
