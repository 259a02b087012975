// Device code of the generic kernels (fwd_kernel, bwd_kernel) and their helpers, shared by the
// translation units that instantiate them (gen_inst.hip, once per direction and activation type,
// so that they compile in parallel) and by kernels.hip (argument structs, element helpers).
#pragma once

#include <algorithm>

#include "ff_internal.h"

namespace ff {
namespace gen {


typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned short u16;

// Accesses to global memory go through global-address-space pointers, so that they compile to
// global rather than flat instructions: a flat access also counts against the LDS counter, and a
// wait for an LDS read would then wait for every global load in flight.
#define FF_GLOBAL __attribute__((address_space(1)))
// (HIP's vector types cannot be accessed through such pointers; they move as raw words.)
typedef unsigned raw2 __attribute__((ext_vector_type(2)));
typedef unsigned raw4 __attribute__((ext_vector_type(4)));
template <int N> struct Raw;
template <> struct Raw<2> { using T = unsigned short; };
template <> struct Raw<4> { using T = unsigned; };
template <> struct Raw<8> { using T = raw2; };
template <> struct Raw<16> { using T = raw4; };
template <class T>
__device__ __forceinline__ T gload(const T* p) {
  using R = typename Raw<sizeof(T)>::T;
  return __builtin_bit_cast(T, *(const FF_GLOBAL R*)p);
}
template <class T>
__device__ __forceinline__ void gstore(T* p, const T& v) {
  using R = typename Raw<sizeof(T)>::T;
  *(FF_GLOBAL R*)p = __builtin_bit_cast(R, v);
}

__device__ __forceinline__ float bf2f(u16 h) { return __uint_as_float((unsigned)h << 16); }

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// Two fp32 values to packed bf16 (a in the low half), round to nearest even: one
// v_cvt_pk_bf16_f32.
__device__ __forceinline__ unsigned pk_bf2(float a, float b) {
  return __builtin_bit_cast(unsigned, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}

// fp32 -> bf16, round to nearest even (NaN kept quiet).
__device__ __forceinline__ u16 f2bf(float f) {
  unsigned u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return (u16)(u >> 16);
}

template <bool BF16>
struct Act;

template <>
struct Act<true> {
  using E = u16;
  static __device__ __forceinline__ float ld(const E* p) { return bf2f(*p); }
  static __device__ __forceinline__ void st(E* p, float v) { *p = (u16)pk_bf2(v, 0.f); }
  static __device__ __forceinline__ f32x4 ld4(const E* p) { return unpack4(*reinterpret_cast<const uint2*>(p)); }
  static __device__ __forceinline__ void st4(E* p, f32x4 v) { *reinterpret_cast<uint2*>(p) = pack4(v); }
  static __device__ __forceinline__ f32x4 gld4(const E* p) { return unpack4(gload(reinterpret_cast<const uint2*>(p))); }
  static __device__ __forceinline__ void gst4(E* p, f32x4 v) { gstore(reinterpret_cast<uint2*>(p), pack4(v)); }
  static __device__ __forceinline__ uint2 pack4(f32x4 v) {
    uint2 w;
    w.x = pk_bf2(v[0], v[1]);
    w.y = pk_bf2(v[2], v[3]);
    return w;
  }
  static __device__ __forceinline__ f32x4 unpack4(uint2 w) {
    return f32x4{bf2f((u16)(w.x & 0xffff)), bf2f((u16)(w.x >> 16)), bf2f((u16)(w.y & 0xffff)),
                 bf2f((u16)(w.y >> 16))};
  }
};

template <>
struct Act<false> {
  using E = float;
  static __device__ __forceinline__ float ld(const E* p) { return *p; }
  static __device__ __forceinline__ void st(E* p, float v) { *p = v; }
  static __device__ __forceinline__ f32x4 ld4(const E* p) { return *reinterpret_cast<const f32x4*>(p); }
  static __device__ __forceinline__ void st4(E* p, f32x4 v) { *reinterpret_cast<f32x4*>(p) = v; }
  static __device__ __forceinline__ f32x4 gld4(const E* p) { return gload(reinterpret_cast<const f32x4*>(p)); }
  static __device__ __forceinline__ void gst4(E* p, f32x4 v) { gstore(reinterpret_cast<f32x4*>(p), v); }
};

// ---------------------------------------------------------------------------------------------
// Frame application.  A "column" is one vector the frame's MFMA matrix M (W2 x W2: the block
// B or B^T, or for factored frames the size-k/4 DFT of the radix-4 split) is applied to: the
// inputs of one (token, block) for dense frames, of one (token, block, residue) for factored
// ones.  Sixteen columns form the B operand of v_mfma_f32_16x16x32_bf16 (16x16x4 for fp32);
// lane l holds column l % 16 and contraction elements 8 (l / 16) .. +7 of each step (4 for fp32).
// Inputs at or past `lim` (the column's storage length) are taken as zero; M is zero there too.

// threadIdx.x, opaque to the optimizer: what a phase derives from it is computed in that phase
// instead of being hoisted out of the backward's tile loop, where it would stay live (and, with
// every phase's share together, spill) through all the other phases.
__device__ __forceinline__ int phase_tid() {
  int t = threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}

template <bool BF16>
struct Mfma;

template <>
struct Mfma<true> {
  using V = bf16x8;
  static constexpr int KS = 32, VL = 8;   // contraction per step, elements per lane and step
  static __device__ __forceinline__ f32x4 step(const V& a, const V& b, f32x4 acc) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
  }
};

template <>
struct Mfma<false> {
  using V = f32x4;
  static constexpr int KS = 16, VL = 4;
  static __device__ __forceinline__ f32x4 step(const V& a, const V& b, f32x4 acc) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[0], b[0], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[1], b[1], acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[2], b[2], acc, 0, 0, 0);
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a[3], b[3], acc, 0, 0, 0);
  }
};

// This lane's contraction inputs of step ks for a column whose storage starts at `in`.
template <bool BF16, bool GSRC>
__device__ __forceinline__ typename Mfma<BF16>::V load_operand(const typename Act<BF16>::E* in, bool ok, int lim,
                                                               int ks, int q) {
  using M = Mfma<BF16>;
  using V = typename M::V;
  V b{};
  const int i0 = ks * M::KS + q * M::VL;
  if (ok && i0 < lim) b = GSRC ? gload(reinterpret_cast<const V*>(in + i0)) : *reinterpret_cast<const V*>(in + i0);
  return b;
}

// Every column c < ncols: epi(c, o, acc) receives outputs o..o+3 (o = 16 mt + 4 (lane / 16)) of
// M applied to the column starting at col(c).  The MT x KT fragments of M stay in registers for
// the whole call; each wave takes every nw-th group of 16 columns and loads the next group's
// inputs while it multiplies the current one.
template <bool BF16, bool GSRC, int MT, int KT, class Col, class Epi>
__device__ __forceinline__ void column_apply_reg(const void* frag, int ncols, int lim, Col col, Epi epi) {
  using M = Mfma<BF16>;
  using V = typename M::V;
  const int lane = phase_tid() & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), nw = blockDim.x >> 6,
            q = lane >> 4;
  const int ngrp = (ncols + 15) / 16;
  if (wave >= ngrp) return;
  const V* fr = reinterpret_cast<const V*>(frag);
  // opaque at every call, so that a caller's loop does not keep the fragments of all its frame
  // applies live across iterations (they would not fit in registers)
  asm volatile("" : "+s"(fr));
  V fa[MT][KT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int ks = 0; ks < KT; ++ks) fa[mt][ks] = gload(&fr[(mt * KT + ks) * 64 + lane]);
  // two operand buffers used in turn (no copies, which would wait for the loads in flight)
  V ba[KT], bb[KT];
  auto load = [&](int g, V (&b)[KT]) {
    const int c = g * 16 + (lane & 15);
    const bool ok = c < ncols;
    const auto* in = col(ok ? c : 0);
#pragma unroll
    for (int ks = 0; ks < KT; ++ks) b[ks] = load_operand<BF16, GSRC>(in, ok, lim, ks, q);
  };
  auto mul = [&](int g, const V (&b)[KT]) {
    f32x4 acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KT; ++ks)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) acc[mt] = M::step(fa[mt][ks], b[ks], acc[mt]);
    const int c = g * 16 + (lane & 15);
    if (c < ncols) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) epi(c, 16 * mt + 4 * q, acc[mt]);
    }
  };
  load(wave, ba);
  for (int g = wave; g < ngrp; g += 2 * nw) {
    if (g + nw < ngrp) load(g + nw, bb);
    mul(g, ba);
    if (g + nw >= ngrp) break;
    if (g + 2 * nw < ngrp) load(g + 2 * nw, ba);
    mul(g + nw, bb);
  }
}

// The same for matrices too large to keep in registers: fragments are read from memory (L1 / L2)
// for every group, four output tiles at a time.  With at most kPre contraction steps a column's
// inputs are all loaded before its first output is stored, so the column may be transformed in
// place (factored frames always qualify: W2 <= 128); longer contractions reload them per output
// chunk and need a separate destination.
template <bool BF16, bool GSRC, class Col, class Epi>
__device__ __forceinline__ void column_apply_mem(const void* frag, int MT, int KT, int ncols, int lim, Col col,
                                                 Epi epi) {
  using M = Mfma<BF16>;
  using V = typename M::V;
  constexpr int kC = 4, kPre = 8;
  const int lane = phase_tid() & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), nw = blockDim.x >> 6,
            q = lane >> 4;
  const int ngrp = (ncols + 15) / 16;
  const V* fr = reinterpret_cast<const V*>(frag);
  const bool pre = KT <= kPre;
  for (int g = wave; g < ngrp; g += nw) {
    const int c = g * 16 + (lane & 15);
    const bool ok = c < ncols;
    const auto* in = col(ok ? c : 0);
    V bp[kPre];
    if (pre) {
#pragma unroll
      for (int ks = 0; ks < kPre; ++ks) bp[ks] = ks < KT ? load_operand<BF16, GSRC>(in, ok, lim, ks, q) : V{};
    }
    for (int mt0 = 0; mt0 < MT; mt0 += kC) {
      f32x4 acc[kC];
#pragma unroll
      for (int j = 0; j < kC; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
      for (int ks = 0; ks < KT; ++ks) {
        V b;
        if (pre) {
          b = bp[0];
#pragma unroll
          for (int j = 1; j < kPre; ++j)
            if (ks == j) b = bp[j];
        } else {
          b = load_operand<BF16, GSRC>(in, ok, lim, ks, q);
        }
#pragma unroll
        for (int j = 0; j < kC; ++j) {
          const V a = gload(&fr[((size_t)min(mt0 + j, MT - 1) * KT + ks) * 64 + lane]);
          if (mt0 + j < MT) acc[j] = M::step(a, b, acc[j]);
        }
      }
      if (ok) {
#pragma unroll
        for (int j = 0; j < kC; ++j)
          if (mt0 + j < MT) epi(c, 16 * (mt0 + j) + 4 * q, acc[j]);
      }
    }
  }
}

// Dispatch on the matrix shape: register-resident for the shapes the frames here produce.
template <bool BF16, bool GSRC, class Col, class Epi>
__device__ __forceinline__ void column_apply(const FrameDev& f, bool synth, int ncols, int lim, Col col, Epi epi) {
  const void* frag = BF16 ? (synth ? f.fs16 : f.fa16) : (synth ? f.fs32 : f.fa32);
  const int KT = BF16 ? f.KT : f.KT4;
#define FF_SHAPE(mt, kt)                                                       \
  case (mt) * 64 + (kt):                                                       \
    column_apply_reg<BF16, GSRC, mt, kt>(frag, ncols, lim, col, epi);          \
    return;
  if constexpr (BF16) {
    switch (f.MT * 64 + KT) {
      FF_SHAPE(1, 1) FF_SHAPE(2, 1) FF_SHAPE(3, 2) FF_SHAPE(4, 2) FF_SHAPE(5, 3) FF_SHAPE(6, 3)
      FF_SHAPE(7, 4) FF_SHAPE(8, 4)
      default: break;
    }
  } else {
    switch (f.MT * 64 + KT) {
      FF_SHAPE(1, 1) FF_SHAPE(2, 2) FF_SHAPE(3, 3) FF_SHAPE(4, 4) FF_SHAPE(5, 5) FF_SHAPE(6, 6)
      default: break;
    }
  }
#undef FF_SHAPE
  column_apply_mem<BF16, GSRC>(frag, f.MT, KT, ncols, lim, col, epi);
}

// ---------------------------------------------------------------------------------------------
// Token-grouped tiles (bf16 activations, frame blocks applied directly, up to 128 wide).  The
// element of token t at token-row offset p (the layout of one token row is unchanged) lives at
// ((t / 4) ldt + p) 4 + t % 4: every coefficient holds four consecutive tokens in 8 bytes, so a
// table row of the sparse phases reads or writes four tokens with one LDS access instead of four.
// The frame applies keep full-width LDS accesses.  A group of 16 MFMA columns is four tokens
// (4 tg .. 4 tg + 3) of four consecutive blocks (4 sq .. 4 sq + 3), column j being token j % 4
// of block j / 4.  Analysis runs the MFMA with its operands swapped (D = X^T M^T: rows are the
// group's columns), so that lane (q, L) ends with the four tokens of block 4 sq + q at output
// coefficient 16 mt + L, one 8-byte LDS write; synthesis reads its operand with
// ds_read_b64_tr_b16.  Token slots past the tile's tokens receive zeros from the analysis (their
// operands are zero), so the sparse phases may read and write whole groups.

typedef short g4_i16x4 __attribute__((ext_vector_type(4)));


// Contraction elements 32 ks + 8 q .. + 7 of column L of a group from a token-grouped LDS tile,
// by two transposed reads: within each 16 lanes the 8-byte chunks form 4 rows of 16 values and
// lane L receives value L of each row.  For read h, lane L supplies element k0 + L / 4 (k0 =
// 32 ks + 8 q + 4 h) of block 4 sq + L % 4, i.e. that block's four tokens, so lane L receives
// elements k0 .. k0 + 3 of its own column.  at(c4, k) is the 8-byte chunk of block 4 sq + c4 at
// element k (k < lim); elements at or past lim are returned as zero.
template <int KT, class At>
__device__ __forceinline__ void g4_tile_operand(At at, int lim, int q, int L, bf16x8 (&b)[KT]) {
#pragma unroll
  for (int ks = 0; ks < KT; ++ks) {
    unsigned w[4];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int k0 = 32 * ks + 8 * q + 4 * h;
      const u16* p = at(L & 3, min(k0 + (L >> 2), lim - 1));
      const raw2 r = __builtin_bit_cast(
          raw2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) g4_i16x4*)(const_cast<u16*>(p))));
      const int nv = lim - k0;   // valid elements of this read (the same in the 16 lanes)
      w[2 * h] = nv >= 2 ? r.x : nv == 1 ? (r.x & 0xffffu) : 0u;
      w[2 * h + 1] = nv >= 4 ? r.y : nv == 3 ? (r.y & 0xffffu) : 0u;
    }
    b[ks] = __builtin_bit_cast(bf16x8, raw4{w[0], w[1], w[2], w[3]});
  }
}

// Every group g < ngrp (token group g / nsq, quad of sub-columns g % nsq; a sub-column is a
// block, or a (block, radix-4 column) of a factored frame): operands from token rows in global
// memory (GSRC: colg(tg, sq, L) is column L's row start, NULL outside the tile) or from the LDS
// tile through at(tg, sq, c4, k).  SWAP gives epi(tg, sq, mt, acc) tokens 0..3 of sub-column
// 4 sq + q at output 16 mt + L (analysis, also in place: a group's operands are all read before
// its outputs are written, and groups are disjoint); otherwise outputs 16 mt + 4 q .. + 3 of
// column L (synthesis).  The fragments stay in registers; each wave takes every nw-th group with
// the next group's operands in flight.
template <bool GSRC, bool SWAP, int MT, int KT, class ColG, class At, class Epi>
__device__ __forceinline__ void column_apply_g4(const void* frag, int ngrp, int nsq, int lim, ColG colg, At at,
                                                Epi epi) {
  using M = Mfma<true>;
  using V = typename M::V;
  const int lane = phase_tid() & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6), nw = blockDim.x >> 6,
            q = lane >> 4, L = lane & 15;
  if (wave >= ngrp) return;
  const V* fr = reinterpret_cast<const V*>(frag);
  asm volatile("" : "+s"(fr));
  V fa[MT][KT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt)
#pragma unroll
    for (int ks = 0; ks < KT; ++ks) fa[mt][ks] = gload(&fr[(mt * KT + ks) * 64 + lane]);
  V ba[KT], bb[KT];
  auto load = [&](int g, V (&b)[KT]) {
    const int tg = g / nsq, sq = g - tg * nsq;
    if constexpr (GSRC) {
      const u16* in = colg(tg, sq, L);
      const bool ok = in != nullptr;
#pragma unroll
      for (int ks = 0; ks < KT; ++ks) b[ks] = load_operand<true, true>(ok ? in : colg(0, 0, 0), ok, lim, ks, q);
    } else {
      g4_tile_operand<KT>([&](int c4, int k) { return at(tg, sq, c4, k); }, lim, q, L, b);
    }
  };
  auto mul = [&](int g, const V (&b)[KT]) {
    f32x4 acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[mt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KT; ++ks)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        acc[mt] = SWAP ? M::step(b[ks], fa[mt][ks], acc[mt]) : M::step(fa[mt][ks], b[ks], acc[mt]);
    const int tg = g / nsq, sq = g - tg * nsq;
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) epi(tg, sq, mt, acc[mt]);
  };
  load(wave, ba);
  for (int g = wave; g < ngrp; g += 2 * nw) {
    if (g + nw < ngrp) load(g + nw, bb);
    mul(g, ba);
    if (g + nw >= ngrp) break;
    if (g + 2 * nw < ngrp) load(g + 2 * nw, ba);
    mul(g + nw, bb);
  }
}

// Dispatch on the matrix shape (MT x KT tiles of M, whose columns have lim elements: W for a
// directly applied block, cs for the DFT of size k/4 of a factored one).
template <bool GSRC, bool SWAP, class ColG, class At, class Epi>
__device__ __forceinline__ void column_apply_g4(const FrameDev& f, bool synth, int ngrp, int nsq, int lim, ColG colg,
                                                At at, Epi epi) {
  const void* frag = synth ? f.fs16 : f.fa16;
#define FF_SHAPE(mt, kt)                                                           \
  case (mt) * 64 + (kt):                                                           \
    column_apply_g4<GSRC, SWAP, mt, kt>(frag, ngrp, nsq, lim, colg, at, epi);      \
    return;
  switch (f.MT * 64 + f.KT) {
    FF_SHAPE(1, 1) FF_SHAPE(2, 1) FF_SHAPE(3, 2) FF_SHAPE(4, 2) FF_SHAPE(5, 3) FF_SHAPE(6, 3)
    FF_SHAPE(7, 4) FF_SHAPE(8, 4)
    default: break;   // not taken: the plan uses these tiles only for matrices up to 128 wide
  }
#undef FF_SHAPE
}

// Two consecutive activations (one complex coordinate) as fp32, and back.
template <bool BF16>
__device__ __forceinline__ float2 ld2(const typename Act<BF16>::E* p) {
  if constexpr (BF16) {
    const unsigned w = *reinterpret_cast<const unsigned*>(p);
    return make_float2(bf2f((u16)(w & 0xffff)), bf2f((u16)(w >> 16)));
  } else {
    return *reinterpret_cast<const float2*>(p);
  }
}
template <bool BF16>
__device__ __forceinline__ void st2(typename Act<BF16>::E* p, float2 v) {
  if constexpr (BF16)
    *reinterpret_cast<unsigned*>(p) = pk_bf2(v.x, v.y);
  else
    *reinterpret_cast<float2*>(p) = v;
}
template <bool BF16>
__device__ __forceinline__ float2 gld2(const typename Act<BF16>::E* p) {
  if constexpr (BF16) {
    const unsigned w = gload(reinterpret_cast<const unsigned*>(p));
    return make_float2(bf2f((u16)(w & 0xffff)), bf2f((u16)(w >> 16)));
  } else {
    return gload(reinterpret_cast<const float2*>(p));
  }
}
template <bool BF16>
__device__ __forceinline__ void gst2(typename Act<BF16>::E* p, float2 v) {
  if constexpr (BF16)
    gstore(reinterpret_cast<unsigned*>(p), pk_bf2(v.x, v.y));
  else
    gstore(reinterpret_cast<float2*>(p), v);
}
__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
// a * (c + i s) and a * (c - i s)
__device__ __forceinline__ float2 cmul(float2 a, float2 w) {
  return make_float2(fmaf(a.x, w.x, -a.y * w.y), fmaf(a.y, w.x, a.x * w.y));
}
__device__ __forceinline__ float2 cmulc(float2 a, float2 w) {
  return make_float2(fmaf(a.x, w.x, a.y * w.y), fmaf(a.y, w.x, -a.x * w.y));
}

// x / d for 0 <= x < 2^24 and 0 < d, with inv = 1 / d in fp32: the product is within one of the
// quotient, which the two corrections make exact.
__device__ __forceinline__ int div_small(int x, int d, float inv) {
  int q = (int)((float)x * inv);
  q -= q * d > x;
  q += (q + 1) * d <= x;
  return q;
}

// The twiddle factors of a single-stage factored frame, copied to LDS (the caller synchronizes).
__device__ __forceinline__ void stage_twiddles(const FrameDev& f, float2* lds) {
  if (f.radix == 1 || f.nst != 1) return;
  const float2* tw = (f.tw);
  for (int i = threadIdx.x; i < 3 * f.k2; i += blockDim.x) lds[i] = gload(&tw[i]);
}

// Radix-4 stage of the factored analysis for every (token, block, b < k2) of a tile:
// Y_a'[b] = w^(-a' b) sum_a X[a k2 + b] (-i)^(a a'), read from the token rows at src and written
// to column a' of the block in the LDS tile (which also gets its padding zeroed).  A thread takes
// kRB items at a time with all their loads issued first.
constexpr int kRB = 8;

template <bool BF16>
__device__ __forceinline__ void radix4_analysis(const FrameDev& f, const float2* tw, int nt,
                                                const typename Act<BF16>::E* src, long ld,
                                                typename Act<BF16>::E* dst, int ldt, int ldb) {
  using E = typename Act<BF16>::E;
  const int k2 = f.k2, W = f.W, cs = f.cs, W2 = f.W2;
  const int per_tok = f.nblk * k2, items = nt * per_tok;
  const float inv_pt = 1.f / (float)per_tok, inv_k2 = 1.f / (float)k2;
  for (int it0 = phase_tid(); it0 < items; it0 += kRB * blockDim.x) {
    float2 x[kRB][4], w[kRB][3];
    int b[kRB];
    E* y[kRB];
#pragma unroll
    for (int u = 0; u < kRB; ++u) {
      const int it = min(it0 + u * (int)blockDim.x, items - 1);   // past the end: a repeat, not stored
      const int t = div_small(it, per_tok, inv_pt), r = it - t * per_tok, blk = div_small(r, k2, inv_k2);
      b[u] = r - blk * k2;
      const E* xp = src + (long)t * ld + blk * W + 2 * b[u];
#pragma unroll
      for (int a = 0; a < 4; ++a) x[u][a] = gld2<BF16>(xp + 2 * a * k2);
#pragma unroll
      for (int a = 0; a < 3; ++a) w[u][a] = tw[a * k2 + b[u]];
      y[u] = dst + t * ldt + blk * ldb + 2 * b[u];
    }
#pragma unroll
    for (int u = 0; u < kRB; ++u) {
      if (it0 + u * (int)blockDim.x >= items) break;
      const float2 s02 = cadd(x[u][0], x[u][2]), d02 = csub(x[u][0], x[u][2]);
      const float2 s13 = cadd(x[u][1], x[u][3]), d13 = csub(x[u][1], x[u][3]);
      const float2 y1 = make_float2(d02.x + d13.y, d02.y - d13.x);   // d02 - i d13
      const float2 y3 = make_float2(d02.x - d13.y, d02.y + d13.x);   // d02 + i d13
      st2<BF16>(y[u], cadd(s02, s13));
      st2<BF16>(y[u] + cs, cmulc(y1, w[u][0]));
      st2<BF16>(y[u] + 2 * cs, cmulc(csub(s02, s13), w[u][1]));
      st2<BF16>(y[u] + 3 * cs, cmulc(y3, w[u][2]));
      if (b[u] == 0)
        for (int a = 0; a < 4; ++a)
          for (int e = W2; e < cs; ++e) Act<BF16>::st(y[u] + a * cs + e, 0.f);
    }
  }
}

// Radix-4 stage of the factored synthesis: X[a k2 + b] = sum_a' i^(a a') w^(a' b) Y'_a'[b] from
// the LDS tile, then out = s X (+ beta out) into the token rows at dst.
template <bool BF16>
__device__ __forceinline__ void radix4_synthesis(const FrameDev& f, const float2* tw, int nt,
                                                 const typename Act<BF16>::E* src, int ldt, int ldb,
                                                 typename Act<BF16>::E* dst, long ld, float s, float beta) {
  using E = typename Act<BF16>::E;
  const int k2 = f.k2, W = f.W, cs = f.cs;
  const int per_tok = f.nblk * k2, items = nt * per_tok;
  const float inv_pt = 1.f / (float)per_tok, inv_k2 = 1.f / (float)k2;
  for (int it0 = phase_tid(); it0 < items; it0 += kRB * blockDim.x) {
    float2 yv[kRB][4], w[kRB][3];
    E* out[kRB];
#pragma unroll
    for (int u = 0; u < kRB; ++u) {
      const int it = min(it0 + u * (int)blockDim.x, items - 1);
      const int t = div_small(it, per_tok, inv_pt), r = it - t * per_tok, blk = div_small(r, k2, inv_k2);
      const int b = r - blk * k2;
      const E* yp = src + t * ldt + blk * ldb + 2 * b;
#pragma unroll
      for (int a = 0; a < 4; ++a) yv[u][a] = ld2<BF16>(yp + a * cs);
#pragma unroll
      for (int a = 0; a < 3; ++a) w[u][a] = tw[a * k2 + b];
      out[u] = dst + (long)t * ld + blk * W + 2 * b;
    }
#pragma unroll
    for (int u = 0; u < kRB; ++u) {
      if (it0 + u * (int)blockDim.x >= items) break;
      const float2 y0 = yv[u][0], y1 = cmul(yv[u][1], w[u][0]), y2 = cmul(yv[u][2], w[u][1]),
                   y3 = cmul(yv[u][3], w[u][2]);
      const float2 s02 = cadd(y0, y2), d02 = csub(y0, y2), s13 = cadd(y1, y3), d13 = csub(y1, y3);
      float2 xo[4];
      xo[0] = cadd(s02, s13);
      xo[2] = csub(s02, s13);
      xo[1] = make_float2(d02.x - d13.y, d02.y + d13.x);   // d02 + i d13
      xo[3] = make_float2(d02.x + d13.y, d02.y - d13.x);   // d02 - i d13
#pragma unroll
      for (int a = 0; a < 4; ++a) {
        float2 v = make_float2(s * xo[a].x, s * xo[a].y);
        if (beta != 0.f) {
          const float2 old = gld2<BF16>(out[u] + 2 * a * k2);
          v.x = fmaf(beta, old.x, v.x);
          v.y = fmaf(beta, old.y, v.y);
        }
        gst2<BF16>(out[u] + 2 * a * k2, v);
      }
    }
  }
}

// Multi-stage factored apply (nst = S >= 2, k = 4^S k2), four lanes per (token, block, residue b):
// the 4^S values x[b + k2 j] of a residue are split over the lanes of a quad by the lowest radix-4
// digit of j, lane q holding v[m] = x[b + k2 (4 m + q)] (4^(S-1) values).  Stages 1 .. S-1 (digits
// a_1 .. a_(S-1), of stride 4^(S-T) in j and 4^(S-T-1) in m) are then local to the lane; a 4 x 4
// transpose within the quad regroups every block of four m into the four values of one group
// {4 m' + a} (lane q then holds m' = 4 g + q, a = 0..3 in v[4 g + a]), and stage S runs locally
// too.  Stage T is decimation in frequency over digit a_T: y_a' = w_k^(-a' n 4^(T-1)) sum_a v_a
// (-i)^(a a'), n = b + k2 (digits of j below a_T); the twiddle is a per-lane base w_k^(a (b +
// k2 q) 4^(T-1)) times w_k^(a 4 k2 lo 4^(T-1)) (lo the digits of m below a_T), which is the same in
// every lane and read through the constant address space.  The output digit a_T' takes a_T's
// place, so position j = (a_1' .. a_S') ends in LDS column j (the base-4 digit reversal of the
// frequency, lds_position), where the MFMA applies the dense DFT of size k2.  fp32 throughout; LDS
// receives the activation type.  The synthesis runs the adjoints in reverse order.  A lane holds 32
// of the 128 values of a three-stage residue, and four times the lanes are at work.
template <int S, int T, bool INV>
__device__ __forceinline__ void msr_stage(float2 (&v)[1 << (2 * S - 2)], int bq, int k2,
                                          const float2* __restrict__ twk) {
  constexpr int NL = 1 << (2 * S - 2);
  constexpr int st = 1 << (2 * (S - T) - 2);   // stride of digit a_T in m (T < S)
  constexpr int tws = 1 << (2 * (T - 1));      // w_{K_{T-1}} = w_k^(4^(T-1))
  float2 wb[3];
#pragma unroll
  for (int a = 1; a < 4; ++a) wb[a - 1] = gload(twk + a * bq * tws);
#pragma unroll
  for (int hi = 0; hi < NL / (4 * st); ++hi)
#pragma unroll
    for (int lo = 0; lo < st; ++lo) {
      const int base = hi * 4 * st + lo;
      float2 w[3];
#pragma unroll
      for (int a = 1; a < 4; ++a) {
        using R = Raw<sizeof(float2)>::T;
        const float2 wu =
            __builtin_bit_cast(float2, *((const __attribute__((address_space(4))) R*)(twk + a * 4 * k2 * lo * tws)));
        w[a - 1] = lo == 0 ? wb[a - 1] : cmul(wb[a - 1], wu);
      }
      float2* x = v + base;
      if constexpr (!INV) {
        const float2 x0 = x[0], x1 = x[st], x2 = x[2 * st], x3 = x[3 * st];
        const float2 s02 = cadd(x0, x2), d02 = csub(x0, x2), s13 = cadd(x1, x3), d13 = csub(x1, x3);
        x[0] = cadd(s02, s13);
        x[st] = cmulc(make_float2(d02.x + d13.y, d02.y - d13.x), w[0]);       // d02 - i d13
        x[2 * st] = cmulc(csub(s02, s13), w[1]);
        x[3 * st] = cmulc(make_float2(d02.x - d13.y, d02.y + d13.x), w[2]);   // d02 + i d13
      } else {   // the adjoint of the stage: twiddles w instead of conj(w), then i^(a a')
        const float2 y0 = x[0], y1 = cmul(x[st], w[0]), y2 = cmul(x[2 * st], w[1]), y3 = cmul(x[3 * st], w[2]);
        const float2 s02 = cadd(y0, y2), d02 = csub(y0, y2), s13 = cadd(y1, y3), d13 = csub(y1, y3);
        x[0] = cadd(s02, s13);
        x[st] = make_float2(d02.x - d13.y, d02.y + d13.x);       // d02 + i d13
        x[2 * st] = csub(s02, s13);
        x[3 * st] = make_float2(d02.x + d13.y, d02.y - d13.x);   // d02 - i d13
      }
    }
}

// Stage S, local after the quad transpose: groups v[4 g .. 4 g + 3] over the lowest digit (n = b).
template <int S, bool INV>
__device__ __forceinline__ void msr_last_stage(float2 (&v)[1 << (2 * S - 2)], int b, const float2* __restrict__ twk) {
  constexpr int NL = 1 << (2 * S - 2);
  constexpr int tws = 1 << (2 * (S - 1));
  float2 w[3];
#pragma unroll
  for (int a = 1; a < 4; ++a) w[a - 1] = gload(twk + a * b * tws);
#pragma unroll
  for (int g = 0; g < NL / 4; ++g) {
    float2* x = v + 4 * g;
    if constexpr (!INV) {
      const float2 s02 = cadd(x[0], x[2]), d02 = csub(x[0], x[2]), s13 = cadd(x[1], x[3]), d13 = csub(x[1], x[3]);
      x[0] = cadd(s02, s13);
      x[1] = cmulc(make_float2(d02.x + d13.y, d02.y - d13.x), w[0]);
      x[2] = cmulc(csub(s02, s13), w[1]);
      x[3] = cmulc(make_float2(d02.x - d13.y, d02.y + d13.x), w[2]);
    } else {
      const float2 y0 = x[0], y1 = cmul(x[1], w[0]), y2 = cmul(x[2], w[1]), y3 = cmul(x[3], w[2]);
      const float2 s02 = cadd(y0, y2), d02 = csub(y0, y2), s13 = cadd(y1, y3), d13 = csub(y1, y3);
      x[0] = cadd(s02, s13);
      x[1] = make_float2(d02.x - d13.y, d02.y + d13.x);
      x[2] = csub(s02, s13);
      x[3] = make_float2(d02.x + d13.y, d02.y - d13.x);
    }
  }
}

// One component of a register exchanged with lane q ^ D of the quad (DPP quad permutation).
template <int D>
__device__ __forceinline__ float quad_swap(float x) {
  constexpr int ctrl = D == 1 ? 0xB1 : 0x4E;   // quad_perm [1,0,3,2] / [2,3,0,1]
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), ctrl, 0xF, 0xF, false));
}

// Lane q's registers v[4 g + i] become lane i's v[4 g + q] (a 4 x 4 transpose per group g): two
// rounds, each swapping one bit of the lane index with the same bit of the register index.
template <int NL>
__device__ __forceinline__ void quad_transpose(float2 (&v)[NL], int q) {
#pragma unroll
  for (int g = 0; g < NL / 4; ++g) {
    float2* x = v + 4 * g;
    const bool o1 = q & 1, o2 = q & 2;
#pragma unroll
    for (int p = 0; p < 2; ++p) {   // bit 0: register pairs (2p, 2p + 1)
      const float2 send = o1 ? x[2 * p] : x[2 * p + 1];
      const float2 got = make_float2(quad_swap<1>(send.x), quad_swap<1>(send.y));
      // selects with constant indices (a store to a selected element would put v in scratch)
      x[2 * p] = o1 ? got : x[2 * p];
      x[2 * p + 1] = o1 ? x[2 * p + 1] : got;
    }
#pragma unroll
    for (int p = 0; p < 2; ++p) {   // bit 1: register pairs (p, p + 2)
      const float2 send = o2 ? x[p] : x[p + 2];
      const float2 got = make_float2(quad_swap<2>(send.x), quad_swap<2>(send.y));
      x[p] = o2 ? got : x[p];
      x[p + 2] = o2 ? x[p + 2] : got;
    }
  }
}

template <bool BF16, int S>
__device__ __forceinline__ void msr_analysis(const FrameDev& f, int nt, const typename Act<BF16>::E* src, long ld,
                                             typename Act<BF16>::E* dst, int ldt, int ldb) {
  using E = typename Act<BF16>::E;
  constexpr int NL = 1 << (2 * S - 2);
  const int k2 = f.k2, W = f.W, cs = f.cs, W2 = f.W2;
  const int per_tok = f.nblk * k2, items = nt * per_tok;
  const float inv_pt = 1.f / (float)per_tok, inv_k2 = 1.f / (float)k2;
  // whole quads: 4 items is a multiple of 4 and so is blockDim
  for (int it4 = phase_tid(); it4 < 4 * items; it4 += blockDim.x) {
    const int q = it4 & 3, it = it4 >> 2;
    const int t = div_small(it, per_tok, inv_pt), r = it - t * per_tok, blk = div_small(r, k2, inv_k2);
    const int b = r - blk * k2;
    const E* xp = src + (long)t * ld + blk * W + 2 * (b + k2 * q);
    float2 v[NL];
#pragma unroll
    for (int m = 0; m < NL; ++m) v[m] = gld2<BF16>(xp + 8 * k2 * m);
    const int bq = b + k2 * q;
    msr_stage<S, 1, false>(v, bq, k2, f.twk);
    if constexpr (S >= 3) msr_stage<S, 2, false>(v, bq, k2, f.twk);
    quad_transpose(v, q);
    msr_last_stage<S, false>(v, b, f.twk);
    // v[4 g + a] is position j = 4 (4 g + q) + a: LDS column j
    E* y = dst + t * ldt + blk * ldb + 2 * b;
#pragma unroll
    for (int g = 0; g < NL / 4; ++g)
#pragma unroll
      for (int a = 0; a < 4; ++a) st2<BF16>(y + (16 * g + 4 * q + a) * cs, v[4 * g + a]);
    if (b == 0)
      for (int g = 0; g < NL / 4; ++g)
        for (int a = 0; a < 4; ++a)
          for (int e = W2; e < cs; ++e) Act<BF16>::st(y + (16 * g + 4 * q + a) * cs + e, 0.f);
  }
}

// Multi-stage factored synthesis: the inverse stages on each (token, block, b) quad read from the
// LDS columns (after the dense DFT^H), then out = s x (+ beta out) into the token rows at dst.
template <bool BF16, int S>
__device__ __forceinline__ void msr_synthesis(const FrameDev& f, int nt, const typename Act<BF16>::E* src, int ldt,
                                              int ldb, typename Act<BF16>::E* dst, long ld, float s, float beta) {
  using E = typename Act<BF16>::E;
  constexpr int NL = 1 << (2 * S - 2);
  const int k2 = f.k2, W = f.W, cs = f.cs;
  const int per_tok = f.nblk * k2, items = nt * per_tok;
  const float inv_pt = 1.f / (float)per_tok, inv_k2 = 1.f / (float)k2;
  for (int it4 = phase_tid(); it4 < 4 * items; it4 += blockDim.x) {
    const int q = it4 & 3, it = it4 >> 2;
    const int t = div_small(it, per_tok, inv_pt), r = it - t * per_tok, blk = div_small(r, k2, inv_k2);
    const int b = r - blk * k2;
    const E* yp = src + t * ldt + blk * ldb + 2 * b;
    float2 v[NL];
#pragma unroll
    for (int g = 0; g < NL / 4; ++g)
#pragma unroll
      for (int a = 0; a < 4; ++a) v[4 * g + a] = ld2<BF16>(yp + (16 * g + 4 * q + a) * cs);
    msr_last_stage<S, true>(v, b, f.twk);
    quad_transpose(v, q);
    const int bq = b + k2 * q;
    if constexpr (S >= 3) msr_stage<S, 2, true>(v, bq, k2, f.twk);
    msr_stage<S, 1, true>(v, bq, k2, f.twk);
    E* out = dst + (long)t * ld + blk * W + 2 * (b + k2 * q);
#pragma unroll
    for (int m = 0; m < NL; ++m) {
      float2 o = make_float2(s * v[m].x, s * v[m].y);
      if (beta != 0.f) {
        const float2 old = gld2<BF16>(out + 8 * k2 * m);
        o.x = fmaf(beta, old.x, o.x);
        o.y = fmaf(beta, old.y, o.y);
      }
      gst2<BF16>(out + 8 * k2 * m, o);
    }
  }
}

// z = P^T x for a tile into a token-grouped LDS tile (frames applied directly): every token slot
// of the tile's groups is written, those past nt with zeros.
__device__ __forceinline__ void analysis_g4(const FrameDev& f, int nt, const u16* src, long ld, u16* dst, int ldt,
                                            int ldb) {
  const int nblk = f.nblk, W = f.W, nsq = (nblk + 3) / 4, ngrp = (nt + 3) / 4 * nsq;
  const int lane = phase_tid() & 63, q = lane >> 4, L = lane & 15;
  column_apply_g4<true, true>(
      f, false, ngrp, nsq, W,
      [&](int tg, int sq, int c) -> const u16* {
        const int t = 4 * tg + (c & 3), b = 4 * sq + (c >> 2);
        return t < nt && b < nblk ? src + (long)t * ld + b * W : nullptr;
      },
      [&](int, int, int, int) -> const u16* { return dst; },
      [&](int tg, int sq, int mt, f32x4 v) {
        const int b = 4 * sq + q, o = 16 * mt + L;
        if (b < nblk && o < W) Act<true>::st4(dst + 4 * (tg * ldt + b * ldb + o), v);
      });
}

// out = s P v (+ beta out) for a tile from a token-grouped LDS tile (frames applied directly).
__device__ __forceinline__ void synthesis_g4(const FrameDev& f, int nt, const u16* src, int ldt, int ldb, u16* dst,
                                             long ld, float s, float beta) {
  const int nblk = f.nblk, W = f.W, nsq = (nblk + 3) / 4, ngrp = (nt + 3) / 4 * nsq;
  const int lane = phase_tid() & 63, q = lane >> 4, L = lane & 15;
  column_apply_g4<false, false>(
      f, true, ngrp, nsq, W, [&](int, int, int) -> const u16* { return src; },
      [&](int tg, int sq, int c4, int k) -> const u16* {
        const int b = min(4 * sq + c4, nblk - 1);
        return src + 4 * (tg * ldt + b * ldb + k);
      },
      [&](int tg, int sq, int mt, f32x4 v) {
        const int t = 4 * tg + (L & 3), b = 4 * sq + (L >> 2), o = 16 * mt + 4 * q;
        if (t < nt && b < nblk && o < W) {
          u16* p = dst + (long)t * ld + b * W + o;
          f32x4 r = v * s;
          if (beta != 0.f) r += beta * Act<true>::gld4(p);
          Act<true>::gst4(p, r);
        }
      });
}

// Radix-4 stage of the factored analysis on a token-grouped tile (single-stage frames): an item is
// (token group, block, residue b < k2); it reads x[a k2 + b] (a = 0..3) of its four tokens from
// the token rows (tokens past nt as zero) and writes the real and the imaginary parts of column
// a' row b, four tokens per 8-byte write.  The columns' padding rows W2 .. cs - 1 are never
// written: the DFT of size k/4 reads its operands only below W2.
constexpr int kRB4 = 2;   // items per thread in flight (16 complex loads each)

__device__ __forceinline__ void radix4_analysis_g4(const FrameDev& f, const float2* tw, int nt, const u16* src,
                                                   long ld, u16* dst, int ldt, int ldb) {
  const int k2 = f.k2, W = f.W, cs = f.cs;
  const int per_tg = f.nblk * k2, items = (nt + 3) / 4 * per_tg;
  const float inv_pt = 1.f / (float)per_tg, inv_k2 = 1.f / (float)k2;
  for (int it0 = phase_tid(); it0 < items; it0 += kRB4 * blockDim.x) {
    float2 x[kRB4][4][4], w[kRB4][3];   // [item][token][a]
    u16* y[kRB4];
#pragma unroll
    for (int u = 0; u < kRB4; ++u) {
      const int it = min(it0 + u * (int)blockDim.x, items - 1);   // past the end: a repeat, not stored
      const int tg = div_small(it, per_tg, inv_pt), r = it - tg * per_tg, blk = div_small(r, k2, inv_k2);
      const int b = r - blk * k2;
#pragma unroll
      for (int i = 0; i < 4; ++i) {   // rows past nt: the last token's, read unconditionally and dropped
        const int t = 4 * tg + i;
        const u16* xp = src + (long)min(t, nt - 1) * ld + blk * W + 2 * b;
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          const float2 v = gld2<true>(xp + 2 * a * k2);
          x[u][i][a] = t < nt ? v : make_float2(0.f, 0.f);
        }
      }
#pragma unroll
      for (int a = 0; a < 3; ++a) w[u][a] = tw[a * k2 + b];
      y[u] = dst + 4 * (tg * ldt + blk * ldb + 2 * b);
    }
#pragma unroll
    for (int u = 0; u < kRB4; ++u) {
      if (it0 + u * (int)blockDim.x >= items) break;
      f32x4 yr[4], yi[4];   // [a'] over the four tokens
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float2* xi = x[u][i];
        const float2 s02 = cadd(xi[0], xi[2]), d02 = csub(xi[0], xi[2]);
        const float2 s13 = cadd(xi[1], xi[3]), d13 = csub(xi[1], xi[3]);
        const float2 o[4] = {cadd(s02, s13), cmulc(make_float2(d02.x + d13.y, d02.y - d13.x), w[u][0]),
                             cmulc(csub(s02, s13), w[u][1]), cmulc(make_float2(d02.x - d13.y, d02.y + d13.x), w[u][2])};
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          yr[a][i] = o[a].x;
          yi[a][i] = o[a].y;
        }
      }
#pragma unroll
      for (int a = 0; a < 4; ++a) {   // the real and imaginary rows are adjacent: one 16-byte write
        const uint2 r = Act<true>::pack4(yr[a]), i = Act<true>::pack4(yi[a]);
        *reinterpret_cast<uint4*>(y[u] + 4 * a * cs) = make_uint4(r.x, r.y, i.x, i.y);
      }
    }
  }
}

// Radix-4 stage of the factored synthesis from a token-grouped tile: an item reads the four tokens
// of column a' row b (real and imaginary parts, one 8-byte read each) and writes out = s x
// (+ beta out) for those of its tokens below nt.
__device__ __forceinline__ void radix4_synthesis_g4(const FrameDev& f, const float2* tw, int nt, const u16* src,
                                                    int ldt, int ldb, u16* dst, long ld, float s, float beta) {
  const int k2 = f.k2, W = f.W, cs = f.cs;
  const int per_tg = f.nblk * k2, items = (nt + 3) / 4 * per_tg;
  const float inv_pt = 1.f / (float)per_tg, inv_k2 = 1.f / (float)k2;
  for (int it0 = phase_tid(); it0 < items; it0 += kRB4 * blockDim.x) {
    f32x4 yr[kRB4][4], yi[kRB4][4];
    float2 w[kRB4][3];
    int tg[kRB4], blk[kRB4], b[kRB4];
#pragma unroll
    for (int u = 0; u < kRB4; ++u) {
      const int it = min(it0 + u * (int)blockDim.x, items - 1);
      tg[u] = div_small(it, per_tg, inv_pt);
      const int r = it - tg[u] * per_tg;
      blk[u] = div_small(r, k2, inv_k2);
      b[u] = r - blk[u] * k2;
      const u16* yp = src + 4 * (tg[u] * ldt + blk[u] * ldb + 2 * b[u]);
#pragma unroll
      for (int a = 0; a < 4; ++a) {   // the real and imaginary rows: one 16-byte read
        const uint4 w = *reinterpret_cast<const uint4*>(yp + 4 * a * cs);
        yr[u][a] = Act<true>::unpack4(make_uint2(w.x, w.y));
        yi[u][a] = Act<true>::unpack4(make_uint2(w.z, w.w));
      }
#pragma unroll
      for (int a = 0; a < 3; ++a) w[u][a] = tw[a * k2 + b[u]];
    }
#pragma unroll
    for (int u = 0; u < kRB4; ++u) {
      if (it0 + u * (int)blockDim.x >= items) break;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int t = 4 * tg[u] + i;
        if (t >= nt) break;
        const float2 y0 = make_float2(yr[u][0][i], yi[u][0][i]);
        const float2 y1 = cmul(make_float2(yr[u][1][i], yi[u][1][i]), w[u][0]);
        const float2 y2 = cmul(make_float2(yr[u][2][i], yi[u][2][i]), w[u][1]);
        const float2 y3 = cmul(make_float2(yr[u][3][i], yi[u][3][i]), w[u][2]);
        const float2 s02 = cadd(y0, y2), d02 = csub(y0, y2), s13 = cadd(y1, y3), d13 = csub(y1, y3);
        const float2 xo[4] = {cadd(s02, s13), make_float2(d02.x - d13.y, d02.y + d13.x), csub(s02, s13),
                              make_float2(d02.x + d13.y, d02.y - d13.x)};
        u16* out = dst + (long)t * ld + blk[u] * W + 2 * b[u];
#pragma unroll
        for (int a = 0; a < 4; ++a) {
          float2 v = make_float2(s * xo[a].x, s * xo[a].y);
          if (beta != 0.f) {
            const float2 old = gld2<true>(out + 2 * a * k2);
            v.x = fmaf(beta, old.x, v.x);
            v.y = fmaf(beta, old.y, v.y);
          }
          gst2<true>(out + 2 * a * k2, v);
        }
      }
    }
  }
}

// The dense DFT of size k/4 applied in place to every (token group, block, radix-4 column) of a
// factored token-grouped tile (single-stage frames: four columns per block), M^T for analysis and
// M for synthesis.  Operands are read below W2 only; outputs up to cs are written (M's rows past
// W2 are zero, so the padding rows receive zeros).
__device__ __forceinline__ void factored_dft_g4(const FrameDev& f, bool synth, int nt, u16* tile, int ldt, int ldb) {
  const int cs = f.cs, nsub = 4 * f.nblk, nsq = f.nblk, ngrp = (nt + 3) / 4 * nsq;
  const int lane = phase_tid() & 63, q = lane >> 4, L = lane & 15;
  column_apply_g4<false, true>(
      f, synth, ngrp, nsq, f.W2, [&](int, int, int) -> const u16* { return tile; },
      [&](int tg, int sq, int c4, int k) -> const u16* {
        const int sub = min(4 * sq + c4, nsub - 1);
        return tile + 4 * (tg * ldt + (sub >> 2) * ldb + (sub & 3) * cs + k);
      },
      [&](int tg, int sq, int mt, f32x4 v) {
        const int sub = 4 * sq + q, o = 16 * mt + L;
        if (o < cs) Act<true>::st4(tile + 4 * (tg * ldt + (sub >> 2) * ldb + (sub & 3) * cs + o), v);
      });
}

// z = P^T x into a token-grouped tile: the block directly, or the radix-4 stage and then the DFT
// of size k/4 in place.
__device__ __forceinline__ void analysis_lds_g4(const FrameDev& f, const float2* tw, int nt, const u16* src, long ld,
                                                u16* dst, int ldt, int ldb) {
  if (f.radix == 1) {
    analysis_g4(f, nt, src, ld, dst, ldt, ldb);
    return;
  }
  radix4_analysis_g4(f, tw, nt, src, ld, dst, ldt, ldb);
  __syncthreads();
  factored_dft_g4(f, false, nt, dst, ldt, ldb);
}

// out = s P v (+ beta out) from a token-grouped tile (factored frames transform it in place first).
__device__ __forceinline__ void synthesis_lds_g4(const FrameDev& f, const float2* tw, int nt, u16* src, int ldt,
                                                 int ldb, u16* dst, long ld, float s, float beta) {
  if (f.radix == 1) {
    synthesis_g4(f, nt, src, ldt, ldb, dst, ld, s, beta);
    return;
  }
  factored_dft_g4(f, true, nt, src, ldt, ldb);
  __syncthreads();
  radix4_synthesis_g4(f, tw, nt, src, ldt, ldb, dst, ld, s, beta);
}

// Zero the padding of every column of a factored tile whose coefficients another phase writes
// (the MFMA reads whole columns of cs elements).  Token-grouped tiles (G4) need none.
template <bool BF16, bool G4 = false>
__device__ __forceinline__ void zero_column_pads(const FrameDev& f, int nt, typename Act<BF16>::E* tile, int ldt,
                                                 int ldb) {
  if (G4 || f.radix == 1 || f.cs == f.W2) return;
  const int padw = f.cs - f.W2, per_tok = f.nblk * f.ncol * padw, items = nt * per_tok;
  for (int it = phase_tid(); it < items; it += blockDim.x) {
    const int t = it / per_tok, r = it - t * per_tok, col = r / padw, e = r - col * padw;
    const int blk = col / f.ncol, a = col - blk * f.ncol;
    Act<BF16>::st(tile + t * ldt + blk * ldb + a * f.cs + f.W2 + e, 0.f);
  }
}

// z = P^T x for a tile: token rows at src (global) -> coefficients in the LDS tile.
// MS: the frame may be applied in several radix-4 stages (nst >= 2); only the kernels built for
// such frames carry that code, so the others keep their register allocation.
// G4: into a token-grouped tile.
template <bool BF16, bool MS = false, bool G4 = false>
__device__ __forceinline__ void analysis_to_lds(const FrameDev& f, const float2* tw, int nt,
                                                const typename Act<BF16>::E* src, long ld, typename Act<BF16>::E* dst,
                                                int ldt, int ldb) {
  using A = Act<BF16>;
  using E = typename A::E;
  if constexpr (G4) {
    static_assert(BF16 && !MS, "token-grouped tiles: bf16, frames in at most one radix-4 stage");
    analysis_lds_g4(f, tw, nt, src, ld, dst, ldt, ldb);
    return;
  }
  const int nblk = f.nblk;
  if (f.radix == 1) {
    const int W = f.W;
    column_apply<BF16, true>(
        f, false, nt * nblk, W,
        [&](int c) {
          const int t = c / nblk;
          return src + (long)t * ld + (c - t * nblk) * W;
        },
        [&](int c, int o, f32x4 v) {
          if (o < W) {
            const int t = c / nblk;
            A::st4(dst + t * ldt + (c - t * nblk) * ldb + o, v);
          }
        });
    return;
  }
  if (!MS || f.nst == 1)
    radix4_analysis<BF16>(f, tw, nt, src, ld, dst, ldt, ldb);
  else if constexpr (MS) {
    if (f.nst == 2)
      msr_analysis<BF16, 2>(f, nt, src, ld, dst, ldt, ldb);
    else
      msr_analysis<BF16, 3>(f, nt, src, ld, dst, ldt, ldb);
  }
  __syncthreads();
  const int cs = f.cs, ncol = f.ncol;
  auto at = [&](int c) -> E* {
    const int tb = c / ncol, t = tb / nblk;
    return dst + t * ldt + (tb - t * nblk) * ldb + (c - tb * ncol) * cs;
  };
  column_apply<BF16, false>(
      f, false, nt * nblk * ncol, cs, [&](int c) -> const E* { return at(c); },
      [&](int c, int o, f32x4 v) {
        if (o < cs) A::st4(at(c) + o, v);
      });
}

// out = s P q (+ beta out) for a tile: coefficients in the LDS tile at src -> token rows at dst.
// Factored frames transform the tile in place first, so src is overwritten.
// G4: from a token-grouped tile.
template <bool BF16, bool MS = false, bool G4 = false>
__device__ __forceinline__ void synthesis_from_lds(const FrameDev& f, const float2* tw, int nt,
                                                   typename Act<BF16>::E* src, int ldt, int ldb,
                                                   typename Act<BF16>::E* dst, long ld, float s, float beta) {
  using A = Act<BF16>;
  using E = typename A::E;
  if constexpr (G4) {
    static_assert(BF16 && !MS, "token-grouped tiles: bf16, frames in at most one radix-4 stage");
    synthesis_lds_g4(f, tw, nt, src, ldt, ldb, dst, ld, s, beta);
    return;
  }
  const int nblk = f.nblk;
  if (f.radix == 1) {
    const int W = f.W;
    column_apply<BF16, false>(
        f, true, nt * nblk, W,
        [&](int c) -> const E* {
          const int t = c / nblk;
          return src + t * ldt + (c - t * nblk) * ldb;
        },
        [&](int c, int o, f32x4 v) {
          if (o < W) {
            const int t = c / nblk;
            E* p = dst + (long)t * ld + (c - t * nblk) * W + o;
            f32x4 r = v * s;
            if (beta != 0.f) r += beta * A::gld4(p);
            A::gst4(p, r);
          }
        });
    return;
  }
  const int cs = f.cs, ncol = f.ncol;
  auto at = [&](int c) -> E* {
    const int tb = c / ncol, t = tb / nblk;
    return src + t * ldt + (tb - t * nblk) * ldb + (c - tb * ncol) * cs;
  };
  column_apply<BF16, false>(
      f, true, nt * nblk * ncol, cs, [&](int c) -> const E* { return at(c); },
      [&](int c, int o, f32x4 v) {
        if (o < cs) A::st4(at(c) + o, v);
      });
  __syncthreads();
  if (!MS || f.nst == 1)
    radix4_synthesis<BF16>(f, tw, nt, src, ldt, ldb, dst, ld, s, beta);
  else if constexpr (MS) {
    if (f.nst == 2)
      msr_synthesis<BF16, 2>(f, nt, src, ldt, ldb, dst, ld, s, beta);
    else
      msr_synthesis<BF16, 3>(f, nt, src, ldt, ldb, dst, ld, s, beta);
  }
}

// Sparse products over a generic stream (GenStream).  Each wave walks its run of stream rows
// with the next kSD rows' entries and coefficients in flight.  Lane l accumulates, for tokens
// tg0 .. tg0 + ntg - 1 of the tile, its slot's entries times the source coefficients (src tile)
// and, at the last row of each slab, stores the sums at its destination in the dst tile.
// BWD (q = C^T u over the columns of C): the walk also yields, per entry, this pass's share of
// dC / s = sum_t u_t[row] z_t[column], z being read from the lane's destination before q is
// written over it; part receives one float per stream element (added to when part_add).
constexpr int kSD = 8;   // stream rows per buffer (two buffers: up to 16 rows in flight)
constexpr int kTG = 8;        // tokens per pass over the stream (a last pass may take 2 to 7)
constexpr int kTGWide = 16;   // tokens per pass while at least that many remain: each pass
                              // starts with a latency-bound load of its first entries

template <bool BF16, bool BWD, bool PART_ADD, int kTG>
__device__ __forceinline__ void stream_products(const GenStream& S, const float* __restrict__ cv,
                                                const typename Act<BF16>::E* src, int ld_src,
                                                typename Act<BF16>::E* dst, int ld_dst, int tg0, int ntg,
                                                bool write_dst, float* part) {
  using A = Act<BF16>;
  const int lane = phase_tid() & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r0 = S.wave_row[wave], r1 = S.wave_row[wave + 1];
  if (r0 >= r1) return;
  const int2* ent = (S.ent);
  src += tg0 * ld_src;
  dst += tg0 * ld_dst;
  // Two buffers of kSD rows, each refilled right after it is consumed, so that the other one's
  // loads stay in flight meanwhile.
  int2 ea[kSD], eb[kSD];
  float ca[kSD], cb[kSD];
  float pa[kSD], pb[kSD];   // PART_ADD: the partial sums to add to, loaded with the entries
  auto load = [&](int r, int2 (&e)[kSD], float (&c)[kSD], float (&pv)[kSD]) {
#pragma unroll
    for (int i = 0; i < kSD; ++i) {
      const int j = min(r + i, r1 - 1) * 64 + lane;   // rows past the run repeat its last one, unused
      e[i] = gload(&ent[j]);
      c[i] = gload(&cv[j]);
      if (BWD && PART_ADD && part) pv[i] = gload(&part[j]);
    }
  };
  // Every row reads kTG token rows without branches (tokens past ntg repeat the last one; their
  // sums are never stored and their dC weights zb are zero), so the reads overlap.
  int tso[kTG], tdo[kTG];
#pragma unroll
  for (int t = 0; t < kTG; ++t) {
    tso[t] = min(t, ntg - 1) * ld_src;
    tdo[t] = min(t, ntg - 1) * ld_dst;
  }
  float acc[kTG], zb[kTG];
#pragma unroll
  for (int t = 0; t < kTG; ++t) acc[t] = zb[t] = 0.f;
  bool start = true;   // the next row begins a slab
  // The source values of row i + 1 are read before row i is processed (the source tile is not
  // written during the walk), alternating between two register sets.
  auto read = [&](const int2& e, float (&x)[kTG]) {
    const int so = e.x & 0x7fffffff;
#pragma unroll
    for (int t = 0; t < kTG; ++t) x[t] = A::ld(src + tso[t] + so);
  };
  // Rows r .. r + n - 1 of a buffer (n = kSD in the main loop, so that its body has no exits).
  auto consume = [&](int r, const int2 (&e)[kSD], const float (&c)[kSD], const float (&pv)[kSD], int n) {
    float xa[kTG], xb[kTG];
    read(e[0], xa);
#pragma unroll
    for (int i = 0; i < kSD; ++i) {
      if (i >= n) break;
      float (&x)[kTG] = (i & 1) ? xb : xa;
      if (i + 1 < kSD && i + 1 < n) read(e[i + 1], (i & 1) ? xa : xb);
      const int d = e[i].y;
      if (BWD && part && start) {
        const int dc0 = max(d, 0);
        float zv[kTG];
#pragma unroll
        for (int t = 0; t < kTG; ++t) zv[t] = A::ld(dst + tdo[t] + dc0);
#pragma unroll
        for (int t = 0; t < kTG; ++t) zb[t] = (t < ntg && d >= 0) ? zv[t] : 0.f;
      }
      start = false;
      float dc = 0.f;
#pragma unroll
      for (int t = 0; t < kTG; ++t) {
        acc[t] = fmaf(c[i], x[t], acc[t]);
        if (BWD) dc = fmaf(x[t], zb[t], dc);
      }
      if (BWD && part) {
        gstore(part + (long)(r + i) * 64 + lane, PART_ADD ? pv[i] + dc : dc);
      }
      if (__builtin_amdgcn_readfirstlane(e[i].x) < 0) {   // the slab's last row (same in every lane)
        if (write_dst && d >= 0) {
#pragma unroll
          for (int t = 0; t < kTG; ++t)
            if (t < ntg) {
              float v = acc[t];
              if constexpr (!BWD && PART_ADD) v += A::ld(dst + t * ld_dst + d);   // a later input chunk
              A::st(dst + t * ld_dst + d, v);
            }
        }
#pragma unroll
        for (int t = 0; t < kTG; ++t) acc[t] = 0.f;
        start = true;
      }
    }
  };
  // whole pairs of buffers first, then the remaining rows
  const int rend = r0 + (r1 - r0) / (2 * kSD) * (2 * kSD);
  load(r0, ea, ca, pa);
  load(r0 + kSD, eb, cb, pb);
  for (int r = r0; r < rend; r += 2 * kSD) {
    consume(r, ea, ca, pa, kSD);
    load(r + 2 * kSD, ea, ca, pa);
    consume(r + kSD, eb, cb, pb, kSD);
    load(r + 3 * kSD, eb, cb, pb);
  }
  if (rend < r1) {
    consume(rend, ea, ca, pa, min(kSD, r1 - rend));
    if (rend + kSD < r1) consume(rend + kSD, eb, cb, pb, r1 - rend - kSD);
  }
}

// One pass over ntg <= kTG tokens with the walk for exactly that many (a single token takes the
// 2-token walk): every token row read per table row is used.
template <bool BF16, bool BWD, bool PART_ADD>
__device__ __forceinline__ void stream_pass(const GenStream& S, const float* __restrict__ cv,
                                            const typename Act<BF16>::E* src, int ld_src, typename Act<BF16>::E* dst,
                                            int ld_dst, int tg, int ntg, bool write_dst, float* part) {
  switch (ntg) {
    case 1:
    case 2: stream_products<BF16, BWD, PART_ADD, 2>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part); break;
    case 3: stream_products<BF16, BWD, PART_ADD, 3>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part); break;
    case 4: stream_products<BF16, BWD, PART_ADD, 4>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part); break;
    case 5: stream_products<BF16, BWD, PART_ADD, 5>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part); break;
    case 6: stream_products<BF16, BWD, PART_ADD, 6>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part); break;
    case 7: stream_products<BF16, BWD, PART_ADD, 7>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part); break;
    default: stream_products<BF16, BWD, PART_ADD, kTG>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part);
  }
}

// The sparse products on token-grouped tiles: the same walk, each table row reading NG groups of
// four tokens (one 8-byte LDS read each) for the pass's tokens tg0 .. tg0 + 4 NG - 1 (tg0 a
// multiple of 4) and writing whole groups at a slab's end.  Token slots past ntg hold zeros in the
// source tile, so their sums are zero; their dC weights zb are zero as well.
template <bool BWD, bool PART_ADD, int NG>
__device__ __forceinline__ void stream_products_g4(const GenStream& S, const float* __restrict__ cv, const u16* src,
                                                   int ld_src, u16* dst, int ld_dst, int tg0, int ntg,
                                                   bool write_dst, float* part) {
  using A = Act<true>;
  constexpr int NT = 4 * NG;
  const int lane = phase_tid() & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r0 = S.wave_row[wave], r1 = S.wave_row[wave + 1];
  if (r0 >= r1) return;
  const int2* ent = (S.ent);
  src += tg0 * ld_src;   // group tg0 / 4 starts at element 4 (tg0 / 4) ld
  dst += tg0 * ld_dst;
  const int gs = 4 * ld_src, gd = 4 * ld_dst;
  int2 ea[kSD], eb[kSD];
  float ca[kSD], cb[kSD];
  float pa[kSD], pb[kSD];
  auto load = [&](int r, int2 (&e)[kSD], float (&c)[kSD], float (&pv)[kSD]) {
#pragma unroll
    for (int i = 0; i < kSD; ++i) {
      const int j = min(r + i, r1 - 1) * 64 + lane;
      e[i] = gload(&ent[j]);
      c[i] = gload(&cv[j]);
      if (BWD && PART_ADD && part) pv[i] = gload(&part[j]);
    }
  };
  float acc[NT], zb[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = zb[t] = 0.f;
  bool start = true;
  auto read = [&](const int2& e, float (&x)[NT]) {
    const int so = 4 * (e.x & 0x7fffffff);
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      const f32x4 v = A::ld4(src + g * gs + so);
#pragma unroll
      for (int i = 0; i < 4; ++i) x[4 * g + i] = v[i];
    }
  };
  auto consume = [&](int r, const int2 (&e)[kSD], const float (&c)[kSD], const float (&pv)[kSD], int n) {
    float xa[NT], xb[NT];
    read(e[0], xa);
#pragma unroll
    for (int i = 0; i < kSD; ++i) {
      if (i >= n) break;
      float (&x)[NT] = (i & 1) ? xb : xa;
      if (i + 1 < kSD && i + 1 < n) read(e[i + 1], (i & 1) ? xa : xb);
      const int d = e[i].y;
      if (BWD && part && start) {
        const int dc0 = 4 * max(d, 0);
#pragma unroll
        for (int g = 0; g < NG; ++g) {
          const f32x4 zv = A::ld4(dst + g * gd + dc0);
#pragma unroll
          for (int k = 0; k < 4; ++k) zb[4 * g + k] = (4 * g + k < ntg && d >= 0) ? zv[k] : 0.f;
        }
      }
      start = false;
      float dc = 0.f;
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        acc[t] = fmaf(c[i], x[t], acc[t]);
        if (BWD) dc = fmaf(x[t], zb[t], dc);
      }
      if (BWD && part) gstore(part + (long)(r + i) * 64 + lane, PART_ADD ? pv[i] + dc : dc);
      if (__builtin_amdgcn_readfirstlane(e[i].x) < 0) {   // the slab's last row (same in every lane)
        if (write_dst && d >= 0) {
#pragma unroll
          for (int g = 0; g < NG; ++g) {
            f32x4 v = f32x4{acc[4 * g], acc[4 * g + 1], acc[4 * g + 2], acc[4 * g + 3]};
            if constexpr (!BWD && PART_ADD) v += A::ld4(dst + g * gd + 4 * d);   // a later input chunk
            A::st4(dst + g * gd + 4 * d, v);
          }
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) acc[t] = 0.f;
        start = true;
      }
    }
  };
  const int rend = r0 + (r1 - r0) / (2 * kSD) * (2 * kSD);
  load(r0, ea, ca, pa);
  load(r0 + kSD, eb, cb, pb);
  for (int r = r0; r < rend; r += 2 * kSD) {
    consume(r, ea, ca, pa, kSD);
    load(r + 2 * kSD, ea, ca, pa);
    consume(r + kSD, eb, cb, pb, kSD);
    load(r + 3 * kSD, eb, cb, pb);
  }
  if (rend < r1) {
    consume(rend, ea, ca, pa, min(kSD, r1 - rend));
    if (rend + kSD < r1) consume(rend + kSD, eb, cb, pb, r1 - rend - kSD);
  }
}

template <bool BWD, bool PART_ADD>
__device__ __forceinline__ void stream_pass_g4(const GenStream& S, const float* __restrict__ cv, const u16* src,
                                               int ld_src, u16* dst, int ld_dst, int tg, int ntg, bool write_dst,
                                               float* part) {
  switch ((ntg + 3) / 4) {
    case 1: stream_products_g4<BWD, PART_ADD, 1>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part); break;
    case 2: stream_products_g4<BWD, PART_ADD, 2>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part); break;
    case 3: stream_products_g4<BWD, PART_ADD, 3>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part); break;
    case 4: stream_products_g4<BWD, PART_ADD, 4>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part); break;
    default: stream_products_g4<BWD, PART_ADD, 5>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part);
  }
}

// All tokens of a token-grouped tile, 20 at a time (each pass starts with a latency-bound load of
// its first entries), the last pass reading only the groups it needs; `add` as for stream_all.
constexpr int kTGWideG4 = 20;

template <bool BWD, bool MAY_ADD>
__device__ __forceinline__ void stream_all_g4(const GenStream& S, const float* __restrict__ cv, const u16* src,
                                              int ld_src, u16* dst, int ld_dst, int nt, bool write_dst, float* part,
                                              bool add) {
  for (int tg = 0; tg < nt; tg += kTGWideG4) {
    const int ntg = min(kTGWideG4, nt - tg);
    if (MAY_ADD && (add || (BWD && tg > 0)))
      stream_pass_g4<BWD, MAY_ADD>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part);
    else
      stream_pass_g4<BWD, false>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part);
  }
}

// All tokens of a tile, kTGWide at a time while that many remain, then kTG, each pass reading
// only as many token rows as it needs.
// `add` (MAY_ADD only): backward, add to the dC partial row (as do the tile's later passes);
// forward, add the sums to the destination (the input side's later chunks).
// G4: on token-grouped tiles.
template <bool BF16, bool BWD, bool MAY_ADD = BWD, bool G4 = false>
__device__ __forceinline__ void stream_all(const GenStream& S, const float* __restrict__ cv,
                                           const typename Act<BF16>::E* src, int ld_src, typename Act<BF16>::E* dst,
                                           int ld_dst, int nt, bool write_dst, float* part, bool add = false) {
  if constexpr (G4) {
    static_assert(BF16, "token-grouped tiles hold bf16");
    stream_all_g4<BWD, MAY_ADD>(S, cv, src, ld_src, dst, ld_dst, nt, write_dst, part, add);
    return;
  }
  for (int tg = 0; tg < nt;) {
    const int ntg = nt - tg >= kTGWide ? kTGWide : min(kTG, nt - tg);
    const bool add_now = MAY_ADD && (add || (BWD && tg > 0));
    if (ntg == kTGWide) {
      if (add_now)
        stream_products<BF16, BWD, MAY_ADD, kTGWide>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part);
      else
        stream_products<BF16, BWD, false, kTGWide>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part);
    } else if (add_now) {
      stream_pass<BF16, BWD, MAY_ADD>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part);
    } else {
      stream_pass<BF16, BWD, false>(S, cv, src, ld_src, dst, ld_dst, tg, ntg, write_dst, part);
    }
    tg += ntg;
  }
}

struct FwdArgs {
  FrameDev fin, fout;
  int T, tt, ldt_in, ldt_out, ldb_in, ldb_out;
  const void* X;
  const void* const* Xs;
  long ldx;
  void* Y;
  void* const* Ys;
  long ldy;
  const float* c;             // coefficients in forward stream order: c (batch: cs[bi]) or
  const float* const* cs;     // ccopy + bi * cstride when the layout differs
  const float* ccopy;
  long cstride;
  float scale, beta;
  GenStream st;
  int nch;              // input-side chunks: blocks chunk_blk[i] .. chunk_blk[i + 1] - 1
  int chunk_blk[kMaxGenChunks + 1];
  // group calls: adapter blockIdx.y's own plan (stream, coefficient copy) and token count
  // (device, clamped to [0, T]; NULL: T)
  const GenDesc* group;
  const int* tokens;
  int g4;               // token-grouped tiles (bf16, frames applied directly, whole input side)
};

__device__ __forceinline__ int group_tokens(const int* tokens, int T, int bi) {
  return tokens ? max(0, min(gload(tokens + bi), T)) : T;
}

// CHUNKED: the input side in a.nch chunks of blocks, v accumulated over them; otherwise whole
// (a.nch == 1), in code of its own.  G4: token-grouped tiles (bf16, whole input side, frames
// applied directly), whose token slots are rounded up to whole groups of four.
template <bool BF16, bool CHUNKED, bool MS = false, bool G4 = false>
__global__ void __launch_bounds__(kFusedThreads) fwd_kernel(FwdArgs a) {
  using A = Act<BF16>;
  using E = typename A::E;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int cap = G4 ? (a.tt + 3) & ~3 : a.tt;   // token slots of a tile
  E* zt = reinterpret_cast<E*>(smem);           // cap x ldt_in   z = P_in^T x (of one chunk)
  E* vt = zt + (size_t)cap * a.ldt_in;          // cap x ldt_out  v = C z
  const int bi = blockIdx.y;
  const E* X = (reinterpret_cast<const E*>(a.Xs ? a.Xs[bi] : a.X));
  E* Y = (reinterpret_cast<E*>(a.Ys ? a.Ys[bi] : a.Y));
  const float* cv = (a.ccopy ? a.ccopy + bi * a.cstride : a.cs ? a.cs[bi] : a.c);
  GenStream st = a.st;
  int T = a.T;
  if (a.group) {   // the adapter's own plan and tokens
    const GenDesc* d = a.group + bi;
    st = d->fwd;
    cv = d->fwd_by_pos ? a.cs[bi] : d->c_fwd;
    T = group_tokens(a.tokens, a.T, bi);
  }
  const int t0 = blockIdx.x * a.tt;
  const int nt = min(a.tt, T - t0);
  if (nt <= 0) return;   // past this adapter's tokens (group calls; uniform)
  X += (long)t0 * a.ldx;
  Y += (long)t0 * a.ldy;

  // twiddle factors of factored frames after the tiles
  float2* tw_in = reinterpret_cast<float2*>(vt + (size_t)cap * a.ldt_out);
  float2* tw_out = tw_in + kTwLdsBytes / 16;
  stage_twiddles(a.fin, tw_in);
  stage_twiddles(a.fout, tw_out);
  if (a.fin.radix != 1 || a.fout.radix != 1) __syncthreads();

  zero_column_pads<BF16, G4>(a.fout, nt, vt, a.ldt_out, a.ldb_out);
  if constexpr (!CHUNKED) {
    // analysis: z = P_in^T x for every (token, input block)
    analysis_to_lds<BF16, MS, G4>(a.fin, tw_in, nt, X, a.ldx, zt, a.ldt_in, a.ldb_in);
    __syncthreads();

    // coefficients: v[a] = sum_{e in row a} c_e z[b_e]
    stream_all<BF16, false, false, G4>(st, cv, zt, a.ldt_in, vt, a.ldt_out, nt, true, nullptr);
  } else {
    for (int ch = 0; ch < a.nch; ++ch) {
      // the chunk's blocks as a frame of their own, at column b0 W of the token rows
      const int b0 = a.chunk_blk[ch];
      FrameDev fc = a.fin;
      fc.nblk = a.chunk_blk[ch + 1] - b0;
      if (ch > 0) __syncthreads();   // the previous chunk's products are done reading z
      analysis_to_lds<BF16, MS, G4>(fc, tw_in, nt, X + (long)b0 * a.fin.W, a.ldx, zt, a.ldt_in, a.ldb_in);
      __syncthreads();

      // v[a] (+)= sum over the chunk's entries of row a of c_e z[b_e]
      GenStream sc = st;
      sc.wave_row += ch * (kGenWaves + 1);
      stream_all<BF16, false, true, G4>(sc, cv, zt, a.ldt_in, vt, a.ldt_out, nt, true, nullptr, ch > 0);
    }
  }
  __syncthreads();

  // synthesis and epilogue: y = beta y + s P_out v
  synthesis_from_lds<BF16, MS, G4>(a.fout, tw_out, nt, vt, a.ldt_out, a.ldb_out, Y, a.ldy, a.scale, a.beta);
}

struct BwdArgs {
  FrameDev fin, fout;
  int T, tt, ldt_in, ldt_out, ldb_in, ldb_out;
  const void* X;
  const void* const* Xs;
  long ldx;
  const void* G;
  const void* const* Gs;
  long ldg;
  void* dX;
  void* const* dXs;
  long lddx;
  const float* ccopy;   // coefficients in backward stream order, [batch][cstride]
  long cstride;
  float scale, beta;
  int want_dx, want_dc;
  GenStream st;
  float* partial;       // dC partial sums [batch][workgroup][cstride]
  long ntiles;
  int nch;              // input-side chunks: blocks chunk_blk[i] .. chunk_blk[i + 1] - 1
  int chunk_blk[kMaxGenChunks + 1];
  // group calls: adapter blockIdx.y's own plan (stream, coefficient copy, partial rows) and
  // token count (device, clamped to [0, T]; NULL: T)
  const GenDesc* group;
  const int* tokens;
  int g4;               // token-grouped tiles (bf16, frames applied directly, whole input side)
};

// CHUNKED: the input side in a.nch chunks of blocks; otherwise whole (a.nch == 1), in code of
// its own (the chunk loop costs registers that the whole-side kernel then spills).  G4 as for the
// forward.
template <bool BF16, bool CHUNKED, bool MS = false, bool G4 = false>
__global__ void __launch_bounds__(kFusedThreads) bwd_kernel(BwdArgs a) {
  using A = Act<BF16>;
  using E = typename A::E;
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int cap = G4 ? (a.tt + 3) & ~3 : a.tt;   // token slots of a tile
  E* ut = reinterpret_cast<E*>(smem);           // cap x ldt_out  u = P_out^T g
  E* zt = ut + (size_t)cap * a.ldt_out;         // cap x ldt_in   z = P_in^T x of one chunk, later q = C^T u
  const int bi = blockIdx.y;
  const E* G0 = reinterpret_cast<const E*>(a.Gs ? a.Gs[bi] : a.G);
  const E* X0 = reinterpret_cast<const E*>(a.Xs ? a.Xs[bi] : a.X);
  E* dX0 = reinterpret_cast<E*>(a.dXs ? a.dXs[bi] : a.dX);
  const float* cv = a.ccopy + bi * a.cstride;
  // one partial row per workgroup, accumulated over the workgroup's tiles
  float* part = a.want_dc ? a.partial + ((long)bi * gridDim.x + blockIdx.x) * a.cstride : nullptr;
  GenStream st = a.st;
  long ntiles = a.ntiles;
  int Tb = a.T;
  if (a.group) {   // the adapter's own plan, workspace and tokens
    const GenDesc* d = a.group + bi;
    st = d->bwd;
    cv = d->c_bwd;
    part = a.want_dc ? d->partial + (long)blockIdx.x * 64 * st.rows : nullptr;
    Tb = group_tokens(a.tokens, a.T, bi);
    ntiles = (Tb + a.tt - 1) / a.tt;
  }

  // twiddle factors of factored frames after the tiles
  float2* tw_in = reinterpret_cast<float2*>(zt + (size_t)cap * a.ldt_in);
  float2* tw_out = tw_in + kTwLdsBytes / 16;
  stage_twiddles(a.fin, tw_in);
  stage_twiddles(a.fout, tw_out);
  if (a.fin.radix != 1 || a.fout.radix != 1) __syncthreads();

  for (long tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const long t0 = tile * a.tt;
    const int nt = (int)min((long)a.tt, (long)Tb - t0);
    if (tile != blockIdx.x) __syncthreads();   // the previous tile's LDS reads are done

    if constexpr (!CHUNKED) {
      // q is written over z and then synthesized from whole columns: their padding must be zero
      zero_column_pads<BF16, G4>(a.fin, nt, zt, a.ldt_in, a.ldb_in);
      analysis_to_lds<BF16, MS, G4>(a.fout, tw_out, nt, G0 + t0 * a.ldg, a.ldg, ut, a.ldt_out, a.ldb_out);
      if (a.want_dc) analysis_to_lds<BF16, MS, G4>(a.fin, tw_in, nt, X0 + t0 * a.ldx, a.ldx, zt, a.ldt_in, a.ldb_in);
      __syncthreads();

      // q[b] = sum_{e in column b} c_e u[a_e] (written over z) and this tile's dC partial sums
      stream_all<BF16, true, true, G4>(st, cv, ut, a.ldt_out, zt, a.ldt_in, nt, a.want_dx, part, tile != blockIdx.x);
      if (!a.want_dx) continue;
      __syncthreads();

      synthesis_from_lds<BF16, MS, G4>(a.fin, tw_in, nt, zt, a.ldt_in, a.ldb_in, dX0 + t0 * a.lddx, a.lddx, a.scale,
                               a.beta);
      continue;
    }
    analysis_to_lds<BF16, MS, G4>(a.fout, tw_out, nt, G0 + t0 * a.ldg, a.ldg, ut, a.ldt_out, a.ldb_out);
    for (int ch = 0; ch < a.nch; ++ch) {
      // the chunk's blocks as a frame of their own, at column b0 W of the token rows
      const int b0 = a.chunk_blk[ch];
      FrameDev fc = a.fin;
      fc.nblk = a.chunk_blk[ch + 1] - b0;
      const long col0 = (long)b0 * a.fin.W;
      if (ch > 0) __syncthreads();   // the previous chunk is done with the z / q tile
      // q is written over z and then synthesized from whole columns: their padding must be zero
      zero_column_pads<BF16, G4>(fc, nt, zt, a.ldt_in, a.ldb_in);
      if (a.want_dc) analysis_to_lds<BF16, MS, G4>(fc, tw_in, nt, X0 + t0 * a.ldx + col0, a.ldx, zt, a.ldt_in, a.ldb_in);
      __syncthreads();

      // q[b] = sum_{e in column b} c_e u[a_e] (written over z) and this tile's dC partial sums
      GenStream sc = st;
      sc.wave_row += ch * (kGenWaves + 1);
      stream_all<BF16, true, true, G4>(sc, cv, ut, a.ldt_out, zt, a.ldt_in, nt, a.want_dx, part, tile != blockIdx.x);
      if (!a.want_dx) continue;
      __syncthreads();

      synthesis_from_lds<BF16, MS, G4>(fc, tw_in, nt, zt, a.ldt_in, a.ldb_in, dX0 + t0 * a.lddx + col0, a.lddx, a.scale,
                               a.beta);
    }
  }
}


// Launch fwd_kernel / bwd_kernel for one activation type (gen_inst.hip); CHUNKED is a.nch > 1.
hipError_t launch_fwd_bf16(const FwdArgs& a, dim3 grid, size_t lds, hipStream_t s);
hipError_t launch_fwd_f32(const FwdArgs& a, dim3 grid, size_t lds, hipStream_t s);
hipError_t launch_bwd_bf16(const BwdArgs& a, dim3 grid, size_t lds, hipStream_t s);
hipError_t launch_bwd_f32(const BwdArgs& a, dim3 grid, size_t lds, hipStream_t s);
// Allow them the largest dynamic LDS allocation (once per process).
hipError_t configure_fwd_bf16();
hipError_t configure_fwd_f32();
hipError_t configure_bwd_bf16();
hipError_t configure_bwd_f32();

}  // namespace gen
}  // namespace ff
