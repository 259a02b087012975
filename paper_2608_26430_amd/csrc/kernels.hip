// HIP kernels of the FrameFT adapter hot path for gfx950 (MI355X).
//
// With k*rho = d the frame P is block diagonal with identical 2k x 2k blocks
// B, so applying P^T (analysis, Sec. 2.1) or P (synthesis) to one token is a
// dense 2k x 2k product per block: over a tile of tokens it is one GEMM whose
// rows are (token, block) pairs.  Those products run on MFMA
// (v_mfma_f32_16x16x32_bf16 for bf16 activations, v_mfma_f32_16x16x4_f32 for
// fp32), with the frame block as the A operand (fragments prepared by
// ff_framegen) and 16 activation rows as the B operand.  The sparse
// coefficient products (v = C z forward, q = C^T u and the support-restricted
// dC = s sum_t u_t z_t^T backward, Appendix A) run on the vector ALUs from
// LDS, where one tile's coefficient vectors are kept whole because the
// support of C is uniformly random.
//
// Kernels:
//   fwd_kernel    x -> z = P_in^T x (LDS) -> v = C z (LDS) -> y = beta y + s P_out v
//   bwd_kernel    g -> u = P_out^T g (LDS), x -> z = P_in^T x (LDS)
//                 -> dC partial per tile: sum_t u[a_e] z[b_e]
//                 -> q = C^T u (LDS, over z) -> dX = beta dX + s P_in q
//   dc_reduce     dC[j] = [dC[j] +] s * sum_tiles partial[tile][j]   (fixed order, per coefficient slot)
//   merge_kernel  W = beta W + s P_out C P_in^T, per (output block, input block)
//                 tile as a sum of rank-1 products of block columns.
#include "gen_kernels.h"

namespace ff {
namespace {

using namespace gen;

// out[bi][j] = c_bi[idx[j]] (0 where idx[j] < 0): coefficients in a stream's order.
__global__ void __launch_bounds__(256) gather_coef(const float* c, const float* const* cs, const int* __restrict__ idx,
                                                   int len, float* out) {
  const int bi = blockIdx.y, j = blockIdx.x * 256 + threadIdx.x;
  if (j >= len) return;
  const float* cv = cs ? cs[bi] : c;
  const int k = idx[j];
  out[(long)bi * len + j] = k >= 0 ? cv[k] : 0.f;
}

// A workgroup owns 64 backward stream elements; each of its 16 waves sums 1/16 of the tiles
// with all loads of a pass in flight, and the 16 sums are combined in a fixed order
// (deterministic) and stored at the element's coefficient slot.  Workgroups past the stream
// zero the coefficient slots that hold no entry (when not accumulating).
constexpr int kDcWaves = 16;
constexpr int kDcBatch = 8;

__global__ void __launch_bounds__(64 * kDcWaves) dc_reduce(const float* __restrict__ partial, long ntiles, int len,
                                                           const int* __restrict__ dst, const int* __restrict__ pad,
                                                           int npad, float scale, int accumulate, float* dC,
                                                           float* const* dCs) {
  __shared__ float red[kDcWaves][64];
  const int bi = blockIdx.y, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  float* out = dCs ? dCs[bi] : dC;
  const int nmain = (len + 63) / 64;
  if ((int)blockIdx.x >= nmain) {
    const int j = ((int)blockIdx.x - nmain) * (int)blockDim.x + threadIdx.x;
    if (!accumulate && j < npad) out[pad[j]] = 0.f;
    return;
  }
  const int e = blockIdx.x * 64 + lane;
  const int ec = min(e, len - 1);   // lanes past the end read the last element and write nothing
  const float* p = partial + (long)bi * ntiles * len + ec;
  float sum = 0.f;
  for (long t0 = w; t0 < ntiles; t0 += (long)kDcWaves * kDcBatch) {
    float v[kDcBatch];
#pragma unroll
    for (int j = 0; j < kDcBatch; ++j) {
      const long t = t0 + (long)j * kDcWaves;
      v[j] = t < ntiles ? p[t * len] : 0.f;
    }
#pragma unroll
    for (int j = 0; j < kDcBatch; ++j) sum += v[j];
  }
  red[w][lane] = sum;
  __syncthreads();
  if (w == 0 && e < len) {
    const int slot = dst[e];
    if (slot < 0) return;
    float tot = 0.f;
#pragma unroll
    for (int i = 0; i < kDcWaves; ++i) tot += red[i][lane];
    const float v = scale * tot;
    out[slot] = accumulate ? out[slot] + v : v;
  }
}

struct MergeArgs {
  const float* Btm;  // output-frame block transposed, W_m x W_m: column a of B_m at Btm + a W_m
  const float* Btn;  // input-frame block transposed,  W_n x W_n
  int Wm, Wn, nblk_in, nsub_r, nsub_c, vec;
  const int* ptr;
  const int4* ent;
  const float* c;
  float scale, beta;
  void* W;
  long ldw;
};

constexpr int kMergeThreads = 256;
constexpr int kMergeTile = 128;                // output rows and columns of a workgroup
constexpr int kMergeChunk = 32;                // entries staged per pass
constexpr int kMergeBatch = 256;               // entries whose columns and s c_e sit in LDS at once
constexpr int kMergeLd = kMergeTile + 16;      // fp32 staging: LDS row stride (floats) per entry; the 4
                                               // entry rows one MFMA operand read touches fall on disjoint banks
constexpr int kMergeBLd = kMergeTile + 16;     // bf16 staging: row stride (bf16) per entry; the 4 rows
                                               // one transposed read touches fall on disjoint banks
typedef short mrg_i16x4 __attribute__((ext_vector_type(4)));

typedef __bf16 mrg_bf16x2 __attribute__((ext_vector_type(2)));
typedef float mrg_f32x2 __attribute__((ext_vector_type(2)));

// Two fp32 values rounded to nearest even bf16, packed low then high (one v_cvt_pk_bf16_f32).
__device__ __forceinline__ unsigned pk_bf16(float a, float b) {
  return __builtin_bit_cast(unsigned, __builtin_convertvector(mrg_f32x2{a, b}, mrg_bf16x2));
}

// The bf16 split x = hi + lo + d of four values (hi = RNE_bf16(x), lo = RNE_bf16(x - hi), x - hi
// exact in fp32, |d| <= 2^-16 |x|), packed into the hi and lo operand words.
__device__ __forceinline__ void split4_bf16(float4 x, uint2& hi, uint2& lo) {
  hi.x = pk_bf16(x.x, x.y);
  hi.y = pk_bf16(x.z, x.w);
  lo.x = pk_bf16(x.x - __uint_as_float(hi.x << 16), x.y - __uint_as_float(hi.x & 0xffff0000u));
  lo.y = pk_bf16(x.z - __uint_as_float(hi.y << 16), x.w - __uint_as_float(hi.y & 0xffff0000u));
}

// W[block R rows, block S columns] = beta W + U V^T over the entries e of the block pair (R, S):
// column e of U is s c_e B_m[:, a'_e], column e of V is B_n[:, b'_e] (the rank-1 terms of
// P_out C P_in^T).  A workgroup owns a 128 x 128 tile of the block pair and each of its waves a
// 64 x 64 quadrant; U and V columns of up to 32 entries at a time are gathered from the transposed
// blocks (coalesced across rows) into LDS and contracted on MFMA.  The MFMA computes the transposed
// tile, so that each lane ends with 4 consecutive columns of one row of W.  The old values of W are
// loaded at the start, so that their reads overlap the contraction.
//  * fp32 W: fp32 operands on v_mfma_f32_16x16x4_f32 (4 entries per instruction), fp32 products and
//    accumulation throughout.
//  * bf16 W: each operand split into bf16 hi and lo parts and the three products hi hi + hi lo +
//    lo hi accumulated on v_mfma_f32_16x16x32_bf16 (32 entries per instruction); each is exact in
//    fp32, so a term u v carries at most 3.01 2^-16 |u v| of error besides the fp32 accumulation,
//    far below the bf16 resolution of the merged weight, at a fifth of the MFMA time.
// Entries past a chunk's end are zero columns.
// MINWG = 3 compiles for three workgroups per CU (at most 168 registers: the accumulators then live
// in the arch VGPRs), which launches with many workgroups use: more of them overlap the W reads,
// contraction and W writes of their tiles (the 70B down projection's merge 464 -> 401 us).  With
// only one or two rounds of workgroups the two-per-CU build (MINWG = 1) is faster.
template <bool BF16W, int MINWG>
__global__ void __launch_bounds__(kMergeThreads, MINWG) merge_kernel(MergeArgs a) {
  constexpr int kF32Bytes = 2 * kMergeChunk * kMergeLd * 4;
  constexpr int kBfBytes = 4 * kMergeChunk * kMergeBLd * 2;
  __shared__ __attribute__((aligned(16))) unsigned char stage[BF16W ? kBfBytes : kF32Bytes];
  __shared__ float es[kMergeBatch];
  __shared__ int ea[kMergeBatch], eb[kMergeBatch];
  const int nsub = a.nsub_r * a.nsub_c;
  const int sub = blockIdx.x % nsub, tile = blockIdx.x / nsub;
  const int R = tile / a.nblk_in, S = tile - R * a.nblk_in;
  const int u0 = (sub / a.nsub_c) * kMergeTile, p0 = (sub % a.nsub_c) * kMergeTile;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, n = lane & 15, q = lane >> 4;
  const int wr = (wv >> 1) * 64, wc = (wv & 1) * 64;   // the wave's quadrant: rows u, columns p
  const bool rmw = a.beta != 0.f;
  using Old = typename std::conditional<BF16W, uint2, float4>::type;
  // lane's outputs: W[u = u0 + wr + 16 i + n][p = p0 + wc + 16 j + 4 q + r], r = 0..3
  auto out_off = [&](int i, int j) -> long {
    return ((long)R * a.Wm + u0 + wr + 16 * i + n) * a.ldw + (long)S * a.Wn + p0 + wc + 16 * j + 4 * q;
  };
  auto live = [&](int i, int j) { return u0 + wr + 16 * i + n < a.Wm && p0 + wc + 16 * j + 4 * q < a.Wn; };
  Old old[4][4];
  if (rmw && a.vec) {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        old[i][j] = Old{};
        if (live(i, j)) {
          if constexpr (BF16W)
            old[i][j] = gload(reinterpret_cast<const uint2*>(reinterpret_cast<const u16*>(a.W) + out_off(i, j)));
          else
            old[i][j] = gload(reinterpret_cast<const float4*>(reinterpret_cast<const float*>(a.W) + out_off(i, j)));
        }
      }
  }

  f32x4 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int beg = a.ptr[tile], end = a.ptr[tile + 1];
  // The tile's entries in batches of up to 256 (usually one): their frame columns and s c_e are put
  // in LDS once per batch (one dependent load chain), then consumed 32 at a time.
  for (int c0 = beg; c0 < end; c0 += kMergeChunk) {
    const int k0 = (c0 - beg) % kMergeBatch;   // position of the chunk in its batch
    const int nch = min(kMergeChunk, end - c0);
    __syncthreads();   // the previous pass has finished reading the staging (and, at a batch start, es / ea / eb)
    if (k0 == 0) {
      const int nb = min(kMergeBatch, end - c0);
      if ((int)threadIdx.x < kMergeBatch) {
        const bool in = (int)threadIdx.x < nb;
        const int4 en = in ? a.ent[c0 + threadIdx.x] : make_int4(0, 0, 0, 0);
        ea[threadIdx.x] = en.x;
        eb[threadIdx.x] = en.y;
        es[threadIdx.x] = in ? a.scale * a.c[en.z] : 0.f;
      }
      __syncthreads();
    }
    if constexpr (BF16W) {
      // entry-major hi / lo rows of U and V (as the fp32 staging, 4 rows or columns per piece)
      u16* uh = reinterpret_cast<u16*>(stage);
      u16* ul = uh + kMergeChunk * kMergeBLd;
      u16* vh = ul + kMergeChunk * kMergeBLd;
      u16* vl = vh + kMergeChunk * kMergeBLd;
#pragma unroll
      for (int it = 0; it < kMergeChunk * 32 / kMergeThreads; ++it) {
        const int x = it * kMergeThreads + threadIdx.x, e = x >> 5, f = (x & 31) * 4;
        float4 uu = make_float4(0.f, 0.f, 0.f, 0.f), vv = uu;
        if (e < nch && u0 + f < a.Wm) {
          const float4 b = *reinterpret_cast<const float4*>(a.Btm + (long)ea[k0 + e] * a.Wm + u0 + f);
          const float sc = es[k0 + e];
          uu = make_float4(sc * b.x, sc * b.y, sc * b.z, sc * b.w);
        }
        if (e < nch && p0 + f < a.Wn) vv = *reinterpret_cast<const float4*>(a.Btn + (long)eb[k0 + e] * a.Wn + p0 + f);
        const int o = e * kMergeBLd + f;
        uint2 h, l;
        split4_bf16(uu, h, l);
        *reinterpret_cast<uint2*>(uh + o) = h;
        *reinterpret_cast<uint2*>(ul + o) = l;
        split4_bf16(vv, h, l);
        *reinterpret_cast<uint2*>(vh + o) = h;
        *reinterpret_cast<uint2*>(vl + o) = l;
      }
      __syncthreads();
      // Operand of lane (n, q): row base + n of U or V at entries 8 q .. 8 q + 7, by two transposed
      // reads (ds_read_b64_tr_b16: within 16 lanes the 8-byte chunks form 4 rows of 16 values and
      // lane i receives value i of each row).  Lane L of the group loads entry 8 q + 4 h + L / 4 at
      // rows base + 4 (L % 4) .. + 3, so lane i receives entries 8 q + 4 h .. + 3 of row base + i.
      const int L = lane & 15;
      auto opnd = [&](const u16* arr, int base) -> bf16x8 {
        unsigned w[4];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const u16* pp = arr + (8 * q + 4 * h + (L >> 2)) * kMergeBLd + base + 4 * (L & 3);
          auto* lp = (__attribute__((address_space(3))) mrg_i16x4*)(const_cast<u16*>(pp));
          const raw2 r = __builtin_bit_cast(raw2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(lp));
          w[2 * h] = r.x;
          w[2 * h + 1] = r.y;
        }
        return __builtin_bit_cast(bf16x8, raw4{w[0], w[1], w[2], w[3]});
      };
      bf16x8 ah[4], al[4], bh[4], bl[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        ah[j] = opnd(vh, wc + 16 * j);
        al[j] = opnd(vl, wc + 16 * j);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        bh[i] = opnd(uh, wr + 16 * i);
        bl[i] = opnd(ul, wr + 16 * i);
      }
      // the small products first; each pass over the 16 accumulators keeps dependent MFMAs apart
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al[j], bh[i], acc[i][j], 0, 0, 0);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[j], bl[i], acc[i][j], 0, 0, 0);
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah[j], bh[i], acc[i][j], 0, 0, 0);
    } else {
      float* us = reinterpret_cast<float*>(stage);
      float* vs = us + kMergeChunk * kMergeLd;
      // entry e's 128 rows of U (and columns of V) as 32 float4 pieces; a thread stages 4 of each
#pragma unroll
      for (int it = 0; it < kMergeChunk * 32 / kMergeThreads; ++it) {
        const int x = it * kMergeThreads + threadIdx.x, e = x >> 5, f = (x & 31) * 4;
        float4 uu = make_float4(0.f, 0.f, 0.f, 0.f), vv = uu;
        if (e < nch && u0 + f < a.Wm) {   // W_m and W_n are multiples of 4: a piece is wholly in or out
          const float4 b = *reinterpret_cast<const float4*>(a.Btm + (long)ea[k0 + e] * a.Wm + u0 + f);
          const float sc = es[k0 + e];
          uu = make_float4(sc * b.x, sc * b.y, sc * b.z, sc * b.w);
        }
        if (p0 + f < a.Wn && e < nch) vv = *reinterpret_cast<const float4*>(a.Btn + (long)eb[k0 + e] * a.Wn + p0 + f);
        *reinterpret_cast<float4*>(&us[e * kMergeLd + f]) = uu;
        *reinterpret_cast<float4*>(&vs[e * kMergeLd + f]) = vv;
      }
      __syncthreads();
      // lane (n, q) supplies V[p = wc + 16 j + n][e0 + q] as the A operand and
      // U[u = wr + 16 i + n][e0 + q] as the B operand
      for (int e0 = 0; e0 < nch; e0 += 4) {
        float av[4], bu[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) av[j] = vs[(e0 + q) * kMergeLd + wc + 16 * j + n];
#pragma unroll
        for (int i = 0; i < 4; ++i) bu[i] = us[(e0 + q) * kMergeLd + wr + 16 * i + n];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int j = 0; j < 4; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[j], bu[i], acc[i][j], 0, 0, 0);
      }
    }
  }
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (!live(i, j)) continue;
      const long off = out_off(i, j);
      f32x4 v = acc[i][j];
      if constexpr (BF16W) {
        u16* w = reinterpret_cast<u16*>(a.W) + off;
        if (a.vec) {
          if (rmw) {
            const uint2 o = old[i][j];
            v[0] = fmaf(a.beta, bf2f((u16)(o.x & 0xffffu)), v[0]);
            v[1] = fmaf(a.beta, bf2f((u16)(o.x >> 16)), v[1]);
            v[2] = fmaf(a.beta, bf2f((u16)(o.y & 0xffffu)), v[2]);
            v[3] = fmaf(a.beta, bf2f((u16)(o.y >> 16)), v[3]);
          }
          gstore(reinterpret_cast<uint2*>(w), make_uint2(pk_bf16(v[0], v[1]), pk_bf16(v[2], v[3])));
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) w[r] = f2bf(rmw ? fmaf(a.beta, bf2f(w[r]), v[r]) : v[r]);
        }
      } else {
        float* w = reinterpret_cast<float*>(a.W) + off;
        if (a.vec) {
          if (rmw) {
            const float4 o = old[i][j];
            v[0] = fmaf(a.beta, o.x, v[0]);
            v[1] = fmaf(a.beta, o.y, v[1]);
            v[2] = fmaf(a.beta, o.z, v[2]);
            v[3] = fmaf(a.beta, o.w, v[3]);
          }
          gstore(reinterpret_cast<float4*>(w), make_float4(v[0], v[1], v[2], v[3]));
        } else {
#pragma unroll
          for (int r = 0; r < 4; ++r) w[r] = rmw ? fmaf(a.beta, w[r], v[r]) : v[r];
        }
      }
    }
}

// Group calls: gather_coef with each adapter's own stream (bwd: backward stream into c_bwd,
// else forward stream into c_fwd).
__global__ void __launch_bounds__(256) gather_coef_group(const float* const* cs, const GenDesc* group, int bwd) {
  const int bi = blockIdx.y;
  const GenDesc* d = group + bi;
  const GenStream st = bwd ? d->bwd : d->fwd;
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= 64 * st.rows) return;
  const int k = gload(st.coef + j);
  gstore((bwd ? d->c_bwd : d->c_fwd) + j, k >= 0 ? gload(cs[bi] + k) : 0.f);
}

// Group calls: dc_reduce over each adapter's own partial rows (one per workgroup that had a tile
// of its tokens), stream and padding slots.
__global__ void __launch_bounds__(64 * kDcWaves) dc_reduce_group(const GenDesc* group, const int* tokens, int T,
                                                                 int tt, int nwg_grid, float scale, int accumulate,
                                                                 float* const* dCs) {
  __shared__ float red[kDcWaves][64];
  const int bi = blockIdx.y, lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const GenDesc* d = group + bi;
  float* out = dCs[bi];
  const int len = 64 * d->bwd.rows, nmain = (len + 63) / 64;
  if ((int)blockIdx.x >= nmain) {
    const int j = ((int)blockIdx.x - nmain) * (int)blockDim.x + threadIdx.x;
    if (!accumulate && j < d->ncoef_pad) gstore(out + gload(d->coef_pad + j), 0.f);
    return;
  }
  const int Tb = group_tokens(tokens, T, bi);
  const long nwg = min((long)(Tb + tt - 1) / tt, (long)nwg_grid);
  const int e = blockIdx.x * 64 + lane;
  const int ec = min(e, len - 1);
  const float* p = d->partial + ec;
  float sum = 0.f;
  for (long t0 = w; t0 < nwg; t0 += (long)kDcWaves * kDcBatch) {
    float v[kDcBatch];
#pragma unroll
    for (int j = 0; j < kDcBatch; ++j) {
      const long t = t0 + (long)j * kDcWaves;
      v[j] = t < nwg ? gload(p + t * len) : 0.f;
    }
#pragma unroll
    for (int j = 0; j < kDcBatch; ++j) sum += v[j];
  }
  red[w][lane] = sum;
  __syncthreads();
  if (w == 0 && e < len) {
    const int slot = gload(d->bwd.coef + e);
    if (slot < 0) return;
    float tot = 0.f;
#pragma unroll
    for (int i = 0; i < kDcWaves; ++i) tot += red[i][lane];
    const float v = scale * tot;
    gstore(out + slot, accumulate ? gload(out + slot) + v : v);
  }
}

// c_plan[j] = c_user[user_of_slot[j]], zero in padding slots.
__global__ void __launch_bounds__(256) coef_to_plan(const float* __restrict__ cu, const int* __restrict__ user_of_slot,
                                                    int nslot, float* __restrict__ cp) {
  const int j = blockIdx.x * 256 + threadIdx.x;
  if (j >= nslot) return;
  const int e = user_of_slot[j];
  cp[j] = e >= 0 ? cu[e] : 0.f;
}

// c_user[e] (+)= c_plan[slot_of_user[e]].
__global__ void __launch_bounds__(256) coef_to_user(const float* __restrict__ cp, const int* __restrict__ slot_of_user,
                                                    int nnz, int accumulate, float* __restrict__ cu) {
  const int e = blockIdx.x * 256 + threadIdx.x;
  if (e >= nnz) return;
  const float v = cp[slot_of_user[e]];
  cu[e] = accumulate ? cu[e] + v : v;
}

void record(hipEvent_t ev, hipStream_t s) {
  if (ev) (void)hipEventRecord(ev, s);
}

}  // namespace

hipError_t configure_kernels() {
  static hipError_t once = [] {
    hipError_t e = hipSuccess;
    for (const hipError_t r : {gen::configure_fwd_bf16(), gen::configure_fwd_f32(), gen::configure_bwd_bf16(),
                               gen::configure_bwd_f32()})
      if (r != hipSuccess) e = r;
    return e;
  }();
  return once;
}

// Coefficients of every adapter in a stream's order: out[bi][j] = c_bi[idx[j]].
hipError_t launch_gather(const float* c, const float* const* cs, const int* idx, int len, int count, float* out,
                         hipStream_t s) {
  const dim3 grid((unsigned)((len + 255) / 256), (unsigned)count);
  hipLaunchKernelGGL(gather_coef, grid, dim3(256), 0, s, c, cs, idx, len, out);
  return hipGetLastError();
}

// Tokens per tile for a call of T tokens on `count` adapters.  The generic kernels run one
// workgroup per CU, so tiles go in rounds of `slots` and a call costs about rounds x (token rows
// its sparse walks read per table row + a fixed part worth kTileOverhead of them).  Of the tile
// sizes up to tt (the plan's LDS limit) the cheapest is taken, the larger one on ties (fewer
// passes over the tables).  Token-grouped tiles (g4) read whole groups of four tokens.
constexpr int kTileOverhead = 2;

int call_tile_tokens(int tt, long T, int count, int slots, bool g4) {
  if (T <= 0 || slots < 1) return tt;
  int best = tt;
  long best_cost = -1;
  for (int t = tt; t >= 1; --t) {
    const long tiles = (T + t - 1) / t * count;
    const long rounds = (tiles + slots - 1) / slots;
    const int rem = t % kTG, walk = g4 ? (t + 3) & ~3 : t - rem + (rem ? std::max(rem, 2) : 0);
    const long cost = rounds * (walk + kTileOverhead);
    if (best_cost < 0 || cost < best_cost) best = t, best_cost = cost;
  }
  return best;
}

hipError_t launch_fwd(const ff_plan* p, int bf16, int count, int T, ActPtrs X, int64_t ldx, const float* c,
                      const float* const* cs, float scale, float beta, ActPtrs Y, int64_t ldy, float* c_saved,
                      hipStream_t s) {
  if (bf16 && p->fast.enabled) return launch_fwd128(p, count, T, X, ldx, c, cs, scale, beta, Y, ldy, c_saved, s);
  FwdArgs a{};
  a.fin = p->fin->dev;
  a.fout = p->fout->dev;
  a.T = T;
  a.tt = call_tile_tokens(p->gen_tile_tokens[bf16], T, count, p->gen_wgs, bf16 && p->gen_g4);
  a.ldt_in = p->gen_ldt_in[bf16];
  a.ldt_out = p->ldt_out[bf16];
  a.nch = p->gen_nch;
  a.g4 = bf16 ? p->gen_g4 : 0;
  for (int i = 0; i <= p->gen_nch; ++i) a.chunk_blk[i] = p->gen_chunk_blk[i];
  a.ldb_in = p->ldb_in;
  a.ldb_out = p->ldb_out;
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
  a.st = p->dev.fwd;
  if (!p->dev.fwd_by_pos) {   // the coefficient layout is another path's: reorder for this stream
    a.cstride = 64L * a.st.rows;
    a.ccopy = p->dev.c_fwd;
    const hipError_t e = launch_gather(c, cs, a.st.coef, (int)a.cstride, count, p->dev.c_fwd, s);
    if (e != hipSuccess) return e;
  }
  const dim3 grid((unsigned)((T + a.tt - 1) / a.tt), (unsigned)count);
  hipEvent_t e0, e1;
  take_timing_events(&e0, &e1);
  record(e0, s);
  const size_t lds = p->gen_lds_bytes[bf16];
  const hipError_t e = bf16 ? gen::launch_fwd_bf16(a, grid, lds, s) : gen::launch_fwd_f32(a, grid, lds, s);
  record(e1, s);
  return e != hipSuccess ? e : hipGetLastError();
}

// Floats of backward scratch (coefficient copy, then dC partial rows) that a single-adapter
// call of T tokens uses on the generic kernels; the partial rows start 256-byte aligned.
size_t gen_bwd_scratch_floats(const ff_plan* p, int bf16, int T, size_t* partial_off) {
  const long cstride = 64L * p->dev.bwd.rows;
  const int tt = call_tile_tokens(p->gen_tile_tokens[bf16], T, 1, p->gen_wgs, bf16 && p->gen_g4);
  const long nwg = std::min<long>((T + tt - 1) / tt, p->gen_rows);
  const size_t off = ((size_t)cstride + 63) / 64 * 64;
  if (partial_off) *partial_off = off;
  return off + (size_t)nwg * (size_t)cstride;
}

size_t bwd_scratch_floats(const ff_plan* p, int bf16, int T) {
  if (T <= 0) return 0;
  if (bf16 && p->fast.enabled) return fast128_bwd_scratch_floats(p, T, nullptr);
  return gen_bwd_scratch_floats(p, bf16, T, nullptr);
}

hipError_t launch_bwd(const ff_plan* p, int bf16, int count, int T, ActPtrs X, int64_t ldx, ActPtrs G,
                      int64_t ldg, const float* c, const float* const* cs, float scale, float beta_dx,
                      ActPtrs dX, int64_t lddx, bool want_dx, int accumulate_dc, float* dC, float* const* dCs,
                      bool want_dc, const float* c_saved, hipStream_t s, const BwdScratch* ws) {
  if (bf16 && p->fast.enabled)
    return launch_bwd128(p, count, T, X, ldx, G, ldg, c, cs, scale, beta_dx, dX, lddx, want_dx, accumulate_dc, dC, dCs,
                         want_dc, c_saved, s, ws);
  if (ws && count != 1) return hipErrorInvalidValue;   // a caller's scratch serves one adapter
  BwdArgs a{};
  a.fin = p->fin->dev;
  a.fout = p->fout->dev;
  a.T = T;
  a.tt = call_tile_tokens(p->gen_tile_tokens[bf16], T, count, p->gen_wgs, bf16 && p->gen_g4);
  a.ldt_in = p->gen_ldt_in[bf16];
  a.ldt_out = p->ldt_out[bf16];
  a.ldb_in = p->ldb_in;
  a.ldb_out = p->ldb_out;
  a.nch = p->gen_nch;
  a.g4 = bf16 ? p->gen_g4 : 0;
  for (int i = 0; i <= p->gen_nch; ++i) a.chunk_blk[i] = p->gen_chunk_blk[i];
  a.X = X.one;
  a.Xs = X.many;
  a.ldx = (long)ldx;
  a.G = G.one;
  a.Gs = G.many;
  a.ldg = (long)ldg;
  a.dX = const_cast<void*>(dX.one);
  a.dXs = const_cast<void* const*>(dX.many);
  a.lddx = (long)lddx;
  a.scale = scale;
  a.beta = beta_dx;
  a.want_dx = want_dx;
  a.want_dc = want_dc;
  a.st = p->dev.bwd;
  a.cstride = 64L * a.st.rows;
  a.ccopy = p->dev.c_bwd;
  a.partial = p->partial;
  if (ws) {   // the caller's scratch instead of the plan's workspace
    size_t off = 0;
    if (gen_bwd_scratch_floats(p, bf16, T, &off) > ws->floats) return hipErrorInvalidValue;
    a.ccopy = ws->base;
    a.partial = ws->base + off;
  }
  const long ntiles = (T + a.tt - 1) / a.tt;
  a.ntiles = ntiles;
  hipEvent_t e0, e1;
  take_timing_events(&e0, &e1);
  const long nwg = std::min<long>(ntiles, p->gen_rows);   // partial rows
  if (T > 0 && (want_dx || want_dc)) {
    // the coefficients feed only q = C^T u: a dC-only call neither reads c_vals (which may then be
    // NULL) nor uses the copy, whose stale values reach no output
    if (want_dx) {
      const hipError_t e = launch_gather(c, cs, a.st.coef, (int)a.cstride, count, const_cast<float*>(a.ccopy), s);
      if (e != hipSuccess) return e;
    }
    const dim3 grid((unsigned)nwg, (unsigned)count);
    record(e0, s);
    const size_t lds = p->gen_lds_bytes[bf16];
    const hipError_t eb = bf16 ? gen::launch_bwd_bf16(a, grid, lds, s) : gen::launch_bwd_f32(a, grid, lds, s);
    record(e1, s);
    if (eb != hipSuccess) return eb;
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  if (want_dc) {
    const int len = (int)a.cstride, nmain = (len + 63) / 64;
    const int npadb = (p->dev.ncoef_pad + 64 * kDcWaves - 1) / (64 * kDcWaves);
    const dim3 grid((unsigned)(nmain + npadb), (unsigned)count);
    hipLaunchKernelGGL(dc_reduce, grid, dim3(64 * kDcWaves), 0, s, a.partial, nwg, len, a.st.coef,
                       p->dev.coef_pad, p->dev.ncoef_pad, scale, accumulate_dc, dC, dCs);
  }
  return hipGetLastError();
}

hipError_t launch_fwd_group(const ff_plan_group* g, int bf16, int T, const int* tokens, const void* const* X,
                            int64_t ldx, const float* const* cs, float scale, float beta, void* const* Y, int64_t ldy,
                            hipStream_t s) {
  const ff_plan* p = g->ref;
  if (bf16 && p->fast.enabled) return launch_fwd128_group(g, T, tokens, X, ldx, cs, scale, beta, Y, ldy, s);
  const unsigned count = (unsigned)g->count;
  FwdArgs a{};
  a.fin = p->fin->dev;
  a.fout = p->fout->dev;
  a.T = T;
  a.tt = call_tile_tokens(p->gen_tile_tokens[bf16], T, (int)count, p->gen_wgs, bf16 && p->gen_g4);
  a.ldt_in = p->gen_ldt_in[bf16];
  a.ldt_out = p->ldt_out[bf16];
  a.nch = p->gen_nch;
  a.g4 = bf16 ? p->gen_g4 : 0;
  for (int i = 0; i <= p->gen_nch; ++i) a.chunk_blk[i] = p->gen_chunk_blk[i];
  a.ldb_in = p->ldb_in;
  a.ldb_out = p->ldb_out;
  a.Xs = X;
  a.ldx = (long)ldx;
  a.Ys = Y;
  a.ldy = (long)ldy;
  a.cs = cs;
  a.scale = scale;
  a.beta = beta;
  a.st = p->dev.fwd;
  a.group = g->gen;
  a.tokens = tokens;
  if (g->any_fwd_gather)   // the layouts are other paths' orders: each adapter's coefficients reordered
    hipLaunchKernelGGL(gather_coef_group, dim3((unsigned)((g->max_gen_fwd + 255) / 256), count), dim3(256), 0, s, cs,
                       g->gen, 0);
  const dim3 grid((unsigned)((T + a.tt - 1) / a.tt), count);
  hipEvent_t e0, e1;
  take_timing_events(&e0, &e1);
  record(e0, s);
  const size_t lds = p->gen_lds_bytes[bf16];
  const hipError_t e = bf16 ? gen::launch_fwd_bf16(a, grid, lds, s) : gen::launch_fwd_f32(a, grid, lds, s);
  record(e1, s);
  return e != hipSuccess ? e : hipGetLastError();
}

hipError_t launch_bwd_group(const ff_plan_group* g, int bf16, int T, const int* tokens, const void* const* X,
                            int64_t ldx, const void* const* G, int64_t ldg, const float* const* cs, float scale,
                            float beta_dx, void* const* dX, int64_t lddx, bool want_dx, int accumulate_dc,
                            float* const* dCs, bool want_dc, hipStream_t s) {
  const ff_plan* p = g->ref;
  if (bf16 && p->fast.enabled)
    return launch_bwd128_group(g, T, tokens, X, ldx, G, ldg, cs, scale, beta_dx, dX, lddx, want_dx, accumulate_dc,
                               dCs, want_dc, s);
  const unsigned count = (unsigned)g->count;
  BwdArgs a{};
  a.fin = p->fin->dev;
  a.fout = p->fout->dev;
  a.T = T;
  a.tt = call_tile_tokens(p->gen_tile_tokens[bf16], T, (int)count, p->gen_wgs, bf16 && p->gen_g4);
  a.ldt_in = p->gen_ldt_in[bf16];
  a.ldt_out = p->ldt_out[bf16];
  a.ldb_in = p->ldb_in;
  a.ldb_out = p->ldb_out;
  a.nch = p->gen_nch;
  a.g4 = bf16 ? p->gen_g4 : 0;
  for (int i = 0; i <= p->gen_nch; ++i) a.chunk_blk[i] = p->gen_chunk_blk[i];
  a.Xs = X;
  a.ldx = (long)ldx;
  a.Gs = G;
  a.ldg = (long)ldg;
  a.dXs = dX;
  a.lddx = (long)lddx;
  a.scale = scale;
  a.beta = beta_dx;
  a.want_dx = want_dx;
  a.want_dc = want_dc;
  a.st = p->dev.bwd;
  a.group = g->gen;
  a.tokens = tokens;
  a.ntiles = (T + a.tt - 1) / a.tt;
  // at most one workgroup per CU and adapter, and no more than every plan has partial rows for
  const long nwg = std::min<long>(a.ntiles, g->min_gen_rows);
  hipEvent_t e0, e1;
  take_timing_events(&e0, &e1);
  if (want_dx && nwg > 0)
    hipLaunchKernelGGL(gather_coef_group, dim3((unsigned)((g->max_gen_bwd + 255) / 256), count), dim3(256), 0, s, cs,
                       g->gen, 1);
  record(e0, s);
  if (nwg > 0) {   // (no tokens: the reduction below writes zeros)
    const size_t lds = p->gen_lds_bytes[bf16];
    const hipError_t eb = bf16 ? gen::launch_bwd_bf16(a, dim3((unsigned)nwg, count), lds, s)
                               : gen::launch_bwd_f32(a, dim3((unsigned)nwg, count), lds, s);
    if (eb != hipSuccess) return eb;
  }
  record(e1, s);
  if (want_dc) {
    const int nmain = (g->max_gen_bwd + 63) / 64;
    const int npadb = (g->max_gen_npad + 64 * kDcWaves - 1) / (64 * kDcWaves);
    hipLaunchKernelGGL(dc_reduce_group, dim3((unsigned)(nmain + npadb), count), dim3(64 * kDcWaves), 0, s, g->gen,
                       tokens, T, a.tt, (int)nwg, scale, accumulate_dc, dCs);
  }
  return hipGetLastError();
}

hipError_t launch_coef_to_plan(const ff_plan* p, const float* c_user, float* c_plan, hipStream_t s) {
  const int n = p->dev.nnz;
  if (n > 0)
    hipLaunchKernelGGL(coef_to_plan, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, c_user, p->dev.user_of_slot,
                       n, c_plan);
  return hipGetLastError();
}

hipError_t launch_coef_to_user(const ff_plan* p, const float* c_plan, float* c_user, int accumulate, hipStream_t s) {
  const int n = p->dev.nnz_user;
  if (n > 0)
    hipLaunchKernelGGL(coef_to_user, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, c_plan, p->dev.slot_of_user,
                       n, accumulate, c_user);
  return hipGetLastError();
}

hipError_t launch_merge(const ff_plan* p, const float* c, float scale, int w_bf16, float beta, void* W,
                        int64_t ldw, hipStream_t s) {
  MergeArgs a{};
  a.Btm = p->fout->dev.Bt32;
  a.Btn = p->fin->dev.Bt32;
  a.Wm = p->fout->dev.W;
  a.Wn = p->fin->dev.W;
  // 4-row / 4-column pieces of the staged columns and of the stores
  if (a.Wm % 4 != 0 || a.Wn % 4 != 0 || !a.Btm || !a.Btn) return hipErrorInvalidValue;
  a.nblk_in = p->fin->dev.nblk;
  a.nsub_r = (a.Wm + kMergeTile - 1) / kMergeTile;
  a.nsub_c = (a.Wn + kMergeTile - 1) / kMergeTile;
  const size_t esz = w_bf16 ? 2 : 4;
  // whole 4-column groups in one access when the base and the row stride keep them aligned
  a.vec = (reinterpret_cast<uintptr_t>(W) % (4 * esz) == 0) && ((size_t)ldw * esz) % (4 * esz) == 0;
  a.ptr = p->dev.mrg_ptr;
  a.ent = p->dev.mrg_ent;
  a.c = c;
  a.scale = scale;
  a.beta = beta;
  a.W = W;
  a.ldw = (long)ldw;
  const long nwg = (long)p->fout->dev.nblk * p->fin->dev.nblk * a.nsub_r * a.nsub_c;
  hipEvent_t e0, e1;
  take_timing_events(&e0, &e1);
  record(e0, s);
  const bool many = nwg >= 6L * p->gen_wgs;   // at least two rounds of three workgroups per CU
  if (w_bf16) {
    if (many)
      hipLaunchKernelGGL((merge_kernel<true, 3>), dim3((unsigned)nwg), dim3(kMergeThreads), 0, s, a);
    else
      hipLaunchKernelGGL((merge_kernel<true, 1>), dim3((unsigned)nwg), dim3(kMergeThreads), 0, s, a);
  } else {
    if (many)
      hipLaunchKernelGGL((merge_kernel<false, 3>), dim3((unsigned)nwg), dim3(kMergeThreads), 0, s, a);
    else
      hipLaunchKernelGGL((merge_kernel<false, 1>), dim3((unsigned)nwg), dim3(kMergeThreads), 0, s, a);
  }
  record(e1, s);
  return hipGetLastError();
}

}  // namespace ff
