// Internal declarations of libframeft: frame and plan objects, the device
// descriptors handed to kernels, and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>

#include <atomic>
#include <cstddef>
#include <cstdint>
#include <vector>

#include "frameft.h"

namespace ff {

// Padding (elements) after each 2k-wide frame block inside an LDS token row,
// so that the 16 rows of an MFMA fragment do not start on the same LDS bank.
constexpr int kBlockPad = 8;
// Largest LDS allocation of one workgroup on gfx950.
constexpr int kMaxLdsBytes = 160 * 1024;
// LDS the generic kernels keep after their tiles for the twiddle factors of factored frames:
// [0, 1536) bytes input frame, [1536, 3072) output frame (3 k2 float2 each, k2 <= 64).
constexpr int kTwLdsBytes = 3072;
// Upper bound on tokens per workgroup tile.
constexpr int kMaxTileTokens = 64;
// Most input-side chunks of a generic-kernel tile.
constexpr int kMaxGenChunks = 64;
// Threads per workgroup of the fused forward / backward kernels.
constexpr int kFusedThreads = 512;

// Device form of a frame: the 2k x 2k block B (every diagonal block of P is B
// when k*rho = d) as MFMA fragments for analysis (P^T) and synthesis (P).
struct FrameDev {
  int d;      // real dimension
  int W;      // block width 2k
  int nblk;   // number of blocks rho/2
  int MT;     // 16-row output tiles, ceil(W/16)
  int KT;     // bf16 contraction steps of 32, ceil(W/32)
  int KT4;    // fp32 contraction steps of 16, ceil(W/16)
  const void* fa16;  // analysis   fragments, bf16x8 [MT][KT][64]
  const void* fs16;  // synthesis  fragments, bf16x8 [MT][KT][64]
  const void* fa32;  // analysis   fragments, f32x4  [MT][KT4][64]
  const void* fs32;  // synthesis  fragments, f32x4  [MT][KT4][64]
  const float* B32;  // B, W x W row-major fp32: B[u][c], u = local coordinate, c = local coefficient
  const float* Bt32; // B transposed (B[u][c] at Bt32[c W + u]) for the merge
  // Factored application (radix == 4): B is the realified unitary DFT of size k = 4 k2, applied
  // as a radix-4 stage on the vector ALUs and a dense realified DFT of size k2 (W2 = 2 k2 wide)
  // on MFMA; the fragments above then hold that W2 x W2 matrix and MT / KT / KT4 refer to it.
  // In LDS a block is stored as four columns of cs elements (cs = W2 rounded up to 8, the
  // rounding zero), column a holding the coefficients of frequencies a, a + 4, a + 8, ...
  // radix == 1: the fragments hold B itself, W2 = cs = W, and a block is stored in order.
  int radix;
  int k2;
  int W2;
  int cs;
  const float2* tw;  // [3][k2]: (cos, sin) of 2 pi (a b mod k) / k for a = 1..3, b < k2
  // Several radix-4 stages (nst = S >= 2, k = 4^S k2): the S decimation-in-frequency stages run in
  // registers, one thread per residue b < k2 holding x[b + k2 j] for j < 4^S, and the block is
  // stored in LDS as ncol = 4^S columns of cs elements; column j holds the sequence whose
  // frequency digits (a_1', ..., a_S') read j = a_1' 4^(S-1) + ... + a_S' (base-4 digit reversal
  // of the frequency).  twk[j] = (cos, sin) of 2 pi j / k for j < k.  nst = 1 is the single stage
  // above (twiddles staged in LDS), nst = 0 the dense block.
  int nst;
  int ncol;
  const float2* twk;
};

// The lift L of a frame P = L^T Pv (every frame the library builds has one).  Pv is the block-
// diagonal frame of the coefficient-space dimension dv = k rho (complex k rho / 2), whose block r is
// the unitary k-point DFT; L (dv x d) places row r of the Spectral Tetris frame F: user complex
// coordinate j of the row's window goes to virtual coordinate r k + (j mod k), weighted by F[r][j].
// The modulation by the k-th roots of unity sees j only through j mod k, so z = Pv^T (L x) is the
// analysis of the requested frame, and y = L^T (Pv v) its synthesis.  With k rho = d, L is the
// identity.  Every user coordinate lies in one or two windows (two inside a T(x) block).
struct LiftDev {
  int dc;                // user complex coordinates, d / 2
  int dvc;               // virtual complex coordinates, k rho / 2
  const int* up_src;     // [dvc] user coordinate feeding virtual coordinate v, -1 for none
  const float* up_w;     // [dvc] its weight F[r][j]
  const int2* dn_v;      // [dc]  the virtual coordinates holding user coordinate j (-1: none)
  const float2* dn_w;    // [dc]  their weights
};

// Position of block-local coefficient c (= 2 i + s: frequency i, real or imaginary part s)
// inside a block's LDS storage.
inline int lds_position(const FrameDev& f, int c) {
  if (f.radix == 1) return c;
  int r = c >> 1, col = 0;
  for (int t = 0; t < f.nst; ++t) {   // frequency digits a_1', a_2', ..., least significant first
    col = 4 * col + (r & 3);
    r >>= 2;
  }
  return col * f.cs + 2 * r + (c & 1);
}
// Elements a block occupies in LDS (before padding).
inline int lds_block_span(const FrameDev& f) { return f.radix == 1 ? f.W : f.ncol * f.cs; }

// Streamed sparse tables of the generic kernels.  Slots (rows of C for v = C z, columns for
// q = C^T u) are sorted by entry count and grouped into slabs of 64; slab s is len_s >= 1 stream
// rows of 64 entries, lane l holding the entries of slot 64 s + l (padding where the slot has
// fewer, or past the last slot).  Entry (row r, lane l) is element 64 r + l.  Each of the
// kGenWaves waves of a workgroup walks a contiguous run of whole slabs.
constexpr int kGenWaves = kFusedThreads / 64;
constexpr int kRowLast = (int)0x80000000u;   // flag in ent.x: the last stream row of its slab
struct GenStream {
  const int2* ent;        // (LDS element offset of the source coefficient within a token row
                          //  | kRowLast, LDS element offset of the lane's destination or -1)
  const int* coef;        // coefficient slot of the entry, -1 for padding
  const int* wave_row;    // [chunks][kGenWaves + 1]: first stream row of each wave, one stream per
                          // input-side chunk
  int rows;               // stream rows; entries = 64 * rows
};

// Device tables of a plan.  "LDS offset" means an element offset inside one token row of an LDS
// tile laid out block by block (block stride ldb = block span + kBlockPad).
struct PlanDev {
  GenStream fwd;             // v = C z: source z, destination v
  GenStream bwd;             // q = C^T u and dC: source u, destination q (over z)
  int fwd_by_pos;            // 1: the coefficient layout is the forward stream's entry order
  const int* coef_pad;       // coefficient slots that hold no entry (dC writes zero there)
  int ncoef_pad;
  // merge: entries bucketed by (output block R, input block S), bucket = R*nblk_in + S.
  const int* mrg_ptr;
  const int4* mrg_ent;       // (local row a', local column b', coefficient slot, 0)
  int mrg_max_bucket;
  int nnz;                   // coefficient slots (nnz plus padding)
  const int* user_of_slot;   // [coefficient slots]: user index of the slot's entry, -1 for padding
  const int* slot_of_user;   // [support entries]: coefficient slot of user entry e
  int nnz_user;              // support entries
  float* c_fwd;              // [batch][64 fwd.rows]: coefficients in forward order (fwd_by_pos == 0)
  float* c_bwd;              // [batch][64 bwd.rows]: coefficients in backward stream order
};

// Entry streams of the 128-wide fused kernels: per pair of adjacent 128-wide
// blocks, `len` rows of 64 lane slots starting at stream row `off`.  Pair entries: (off, len,
// mask_off, first mask word).  The streams run in rounds whose last rows are marked in a bit
// mask (bit r of word r / 32 at `mask_off`; the first word is also kept in the entry).
struct FastPlanDev {
  int enabled = 0;
  const int4* fwd_pl = nullptr;       // v = C z, per output pair
  const uint32_t* fwd_st = nullptr;   // slot words; slot (row r, lane l) is coefficient slot 64 r + l
  const int* pad = nullptr;           // coefficient slots that hold no entry
  int npad = 0;
  const int4* bwd_pl = nullptr;       // dC and q = C^T u, per input pair
  const uint32_t* fwd_em = nullptr;   // round-end masks of the forward streams
  const uint32_t* bwd_em = nullptr;   // round-end masks of the backward streams
  const int* bwd_pad = nullptr;       // backward slots that hold no entry
  int nbpad = 0;
  const uint32_t* bwd_st = nullptr;   // slot words
  const uint32_t* bwd_dst = nullptr;  // per backward slot: its coefficient slot, ~0 for padding
  int bwd_slots = 0;                  // 64 * backward stream rows = dC partials per tile
  float* coef_bwd = nullptr;          // [batch][bwd_slots + 256]: c in backward slot order
  const int* bwd_pos = nullptr;       // per coefficient slot: its backward slot (padding: bwd_slots)
  int coef_slots = 0;
  int bwd16 = 0;   // the backward runs 16-token tiles (slot words address 32-byte rows)
};

// One adapter's view of its plan inside a plan group (ff_plan_group): the tables and the
// workspace (batch slot 0 of the plan's own) that the group kernels read per adapter.
struct FastDesc {   // fused 128-wide kernels
  const int4* fwd_pl;
  const uint32_t* fwd_st;
  const uint32_t* fwd_em;
  const int4* bwd_pl;
  const uint32_t* bwd_st;
  const uint32_t* bwd_em;
  const uint32_t* bwd_dst;
  const int* pad;
  const int* bwd_pad;
  const int* bwd_pos;
  float* coef;      // coefficients in backward slot order, bwd_slots + 256
  float* partial;   // dC partials, [tile][bwd_slots + 256]
  int npad, nbpad, slots, coef_slots;
  int bwd16;        // this plan's backward runs 16-token tiles (else 8)
};
struct GenDesc {    // generic kernels
  GenStream fwd, bwd;
  const int* coef_pad;
  float* c_fwd;     // coefficients in forward stream order (when the layout is not that order)
  float* c_bwd;     // coefficients in backward stream order
  float* partial;   // dC partial rows, [workgroup][64 bwd.rows]
  int fwd_by_pos, ncoef_pad;
};

}  // namespace ff

struct ff_frame {
  std::atomic<int> refs{1};
  int64_t d = 0, k = 0, rho = 0;
  int64_t dv = 0;          // coefficient-space dimension k rho (the kernels' frame works in it)
  bool lifted = false;     // k rho != d: P = L^T Pv with a lift L that is not the identity
  ff::LiftDev lift{};
  int device = 0;
  std::vector<double> B;   // W x W fp64 block on the host
  bool transpose_is_sign_flip = false;   // B^T == D B D exactly, D = diag((-1)^i)
  bool half_shift_sign = false;          // B[u + W/2][c] == (-1)^(c/2) B[u][c]
  void* dev_mem = nullptr;
  ff::FrameDev dev{};
};

struct ff_plan {
  ff_frame* fin = nullptr;
  ff_frame* fout = nullptr;
  int64_t nnz = 0, max_tokens = 0, max_batch = 1;
  int64_t coef_slots = 0;          // length of c_vals / dC arrays: nnz plus padding slots
  int device = 0;
  int ldb_in = 0, ldb_out = 0;     // LDS block strides (elements)
  int ldt_in[2] = {0, 0};          // LDS token strides of the input-side tile, [FF_F32], [FF_BF16]
  int ldt_out[2] = {0, 0};
  int tile_tokens[2] = {0, 0};     // tokens per fused-kernel tile
  size_t lds_bytes[2] = {0, 0};
  // Generic-kernel tiles with the input side in chunks: the output side (v, u) whole and z / q
  // one chunk of input blocks at a time, chunk i = blocks gen_chunk_blk[i] .. gen_chunk_blk[i + 1] - 1
  // (one chunk: the whole-side geometry above).
  int gen_nch = 1;
  int gen_chunk_blk[ff::kMaxGenChunks + 1] = {};
  int gen_ldt_in[2] = {0, 0};      // LDS token stride of the input-side chunk tile
  int gen_tile_tokens[2] = {0, 0};
  size_t gen_lds_bytes[2] = {0, 0};
  // bf16 generic kernels on token-grouped tiles (four tokens per coefficient; tiles a multiple of
  // four tokens): frames applied directly (blocks up to 128 wide) or in one radix-4 stage, no lift.
  int gen_g4 = 0;
  int gen_wgs = 1;                 // compute units: resident workgroups of the generic kernels
  int gen_rows = 1;                // dC partial rows per adapter = most workgroups of the generic backward
  float* partial = nullptr;        // dC partial sums per tile (layout depends on the kernels)
  // Merge through the backward (frames with a lift): mrg_rows output rows at a time, their lifted
  // unit vectors as fp32 "upstream gradients" (mrg_rows x m) and the fp32 rows before they are
  // lifted back into the weight (mrg_rows x n).
  int mrg_rows = 0;
  float* mrg_g = nullptr;
  float* mrg_out = nullptr;
  // Frames with a lift (k rho != d on either side): every call lifts its inputs into fp32 staging
  // rows of the coefficient-space width, runs the kernels there in fp32 and lifts the results
  // back.  lift_x: max_tokens x dv_in (X), lift_g: max_tokens x dv_out (G, or the forward's output
  // before the lift), lift_dx: max_tokens x dv_in (dX before the lift).
  bool lifted = false;
  float* lift_x = nullptr;
  float* lift_g = nullptr;
  float* lift_dx = nullptr;
  size_t workspace_bytes = 0;
  void* dev_mem = nullptr;
  ff::PlanDev dev{};
  ff::FastPlanDev fast{};
  std::vector<int64_t> user_order;  // user index of each coefficient slot, -1 for padding
};

// Adapters with their own supports over one frame pair (per-layer masks, tenants), run together:
// plans[i] serves adapter i.  The plans must outlive the group and agree on everything but the
// support (frames, kernel path, tile geometry).
struct ff_plan_group {
  int64_t count = 0;
  std::vector<const ff_plan*> plans;
  const ff_plan* ref = nullptr;   // plans[0]: the shared geometry
  int64_t max_tokens = 0;         // smallest max_tokens of the plans
  int max_fast_items = 0;         // largest coef_slots + nbpad (fused coefficient scatter)
  int max_fast_slots = 0;         // largest bwd_slots
  int max_fast_npad = 0;
  int fast16 = 0, fast8 = 0;      // some plan's fused backward runs 16-token / 8-token tiles
  int max_gen_fwd = 0;            // largest 64 fwd.rows / 64 bwd.rows (generic streams)
  int max_gen_bwd = 0;
  int max_gen_npad = 0;
  int any_fwd_gather = 0;         // some plan's layout is not its forward stream's order
  int min_gen_rows = 0;           // fewest dC partial rows (generic backward) of any plan
  void* dev_mem = nullptr;
  const ff::FastDesc* fast = nullptr;   // [count], device
  const ff::GenDesc* gen = nullptr;     // [count], device
};

namespace ff {

// Error reporting (capi.cpp): remember a message for ff_last_error and return s.
ff_status fail(ff_status s, const char* fmt, ...);
void clear_error();

// One-shot kernel timing events armed by ff_time_next_kernel.
void take_timing_events(hipEvent_t* start, hipEvent_t* stop);

// Launchers (kernels.hip).  Arguments are validated by the caller.
struct ActPtrs {          // one tensor: either a single pointer or a device array of pointers
  const void* one;
  const void* const* many;
};

// c_saved: the backward-ordered coefficient copy of the 128-wide path (written by the
// forward, read by the backward instead of reordering c itself); NULL elsewhere.
hipError_t launch_fwd(const ff_plan* p, int bf16, int count, int T, ActPtrs X, int64_t ldx,
                      const float* c, const float* const* cs, float scale, float beta,
                      ActPtrs Y, int64_t ldy, float* c_saved, hipStream_t s);
// Scratch for a single-adapter backward supplied by the caller (ff_adapter_bwd_noalloc) in place of
// the plan's workspace: `floats` floats at `base`, 256-byte aligned, holding the coefficients in
// the backward's order and then the dC partial sums.  Its contents on entry do not matter.
struct BwdScratch {
  float* base;
  size_t floats;
};
// Floats of BwdScratch a single-adapter backward of T tokens needs (0 for T = 0).
size_t bwd_scratch_floats(const ff_plan* p, int bf16, int T);
size_t fast128_bwd_scratch_floats(const ff_plan* p, int T, size_t* partial_off);
hipError_t launch_bwd(const ff_plan* p, int bf16, int count, int T, ActPtrs X, int64_t ldx,
                      ActPtrs G, int64_t ldg, const float* c, const float* const* cs, float scale,
                      float beta_dx, ActPtrs dX, int64_t lddx, bool want_dx, int accumulate_dc,
                      float* dC, float* const* dCs, bool want_dc, const float* c_saved, hipStream_t s,
                      const BwdScratch* ws = nullptr);
hipError_t launch_merge(const ff_plan* p, const float* c, float scale, int w_bf16, float beta,
                        void* W, int64_t ldw, hipStream_t s);
// Group calls: adapter i runs plans[i] on tokens[i] (device int32, clamped to [0, T]; NULL: all T)
// of its own X / Y / G / dX / c / dC (device pointer arrays).
hipError_t launch_fwd_group(const ff_plan_group* g, int bf16, int T, const int* tokens, const void* const* X,
                            int64_t ldx, const float* const* cs, float scale, float beta, void* const* Y, int64_t ldy,
                            hipStream_t s);
hipError_t launch_bwd_group(const ff_plan_group* g, int bf16, int T, const int* tokens, const void* const* X,
                            int64_t ldx, const void* const* G, int64_t ldg, const float* const* cs, float scale,
                            float beta_dx, void* const* dX, int64_t lddx, bool want_dx, int accumulate_dc,
                            float* const* dCs, bool want_dc, hipStream_t s);
hipError_t launch_fwd128_group(const ff_plan_group* g, int T, const int* tokens, const void* const* X, int64_t ldx,
                               const float* const* cs, float scale, float beta, void* const* Y, int64_t ldy,
                               hipStream_t s);
hipError_t launch_bwd128_group(const ff_plan_group* g, int T, const int* tokens, const void* const* X, int64_t ldx,
                               const void* const* G, int64_t ldg, const float* const* cs, float scale, float beta_dx,
                               void* const* dX, int64_t lddx, bool want_dx, int accumulate_dc, float* const* dCs,
                               bool want_dc, hipStream_t s);
// Calls on plans with a lift (lift.hip): the same contracts as launch_fwd / launch_bwd /
// launch_merge for one adapter, in the user's dimensions.
hipError_t launch_fwd_lifted(const ff_plan* p, int bf16, int T, const void* X, int64_t ldx, const float* c,
                             float scale, float beta, void* Y, int64_t ldy, hipStream_t s);
hipError_t launch_bwd_lifted(const ff_plan* p, int bf16, int T, const void* X, int64_t ldx, const void* G,
                             int64_t ldg, const float* c, float scale, float beta_dx, void* dX, int64_t lddx,
                             bool want_dx, int accumulate_dc, float* dC, bool want_dc, hipStream_t s,
                             const BwdScratch* ws = nullptr);
hipError_t launch_merge_lifted(const ff_plan* p, const float* c, float scale, int w_bf16, float beta, void* W,
                               int64_t ldw, hipStream_t s);
// Generic-kernel tile size of a call (kernels.hip), shared by single, batched and group calls.
int call_tile_tokens(int tt, long T, int count, int slots, bool g4);

// Coefficient vectors between the caller's support order and the plan layout (Algorithm 1,
// step 4): to_plan writes every slot (zero in padding slots), to_user every user entry (added to
// the old value when accumulate).
hipError_t launch_coef_to_plan(const ff_plan* p, const float* c_user, float* c_plan, hipStream_t s);
hipError_t launch_coef_to_user(const ff_plan* p, const float* c_plan, float* c_user, int accumulate,
                               hipStream_t s);
// Set the per-kernel dynamic LDS limits once per process.
hipError_t configure_kernels();

// 128-wide fused path (kernels_w128.hip).
hipError_t configure_fast128();
size_t fast128_lds_bytes(int nblk);
// Floats per tile of the fused backward's dC workspace for a plan with `bwd_slots` slots.
size_t fast128_partial_floats(size_t bwd_slots);
// LDS of the 16-token backward for an output side of nblk_out 128-wide blocks.
size_t fast16_lds_bytes(int nblk_out);
hipError_t launch_fwd128(const ff_plan* p, int count, int T, ActPtrs X, int64_t ldx, const float* c,
                         const float* const* cs, float scale, float beta, ActPtrs Y, int64_t ldy, float* c_saved,
                         hipStream_t s);
hipError_t launch_bwd128(const ff_plan* p, int count, int T, ActPtrs X, int64_t ldx, ActPtrs G, int64_t ldg,
                         const float* c, const float* const* cs, float scale, float beta_dx, ActPtrs dX,
                         int64_t lddx, bool want_dx, int accumulate_dc, float* dC, float* const* dCs, bool want_dc,
                         const float* c_saved, hipStream_t s, const BwdScratch* ws);
constexpr int kFastTileTokens = 8;

// Slot words of the 128-wide kernels' entry streams: restart flag (bit 0: the lane's row ends
// with the round that ends at this slot), valid flag (bit 1: the slot holds an entry;
// padding slots have zero coefficients), the byte offset of the source row in the LDS
// coefficient array (rows of 16 bytes; bits 4..19) and the byte offset of the lane's current
// row in the pair tile (rows of 32 bytes, one per coefficient, holding both blocks' 8 tokens;
// bits 20..31).  Stream row r, lane l of a pair whose rows start at `off` (a multiple of 4)
// is slot 64 off + 256 (r / 4) + 4 l + r % 4: each lane's four consecutive rows are
// contiguous, so a wave loads them with one 16-byte load per lane.
constexpr uint32_t kSlotEnd = 1u;
constexpr uint32_t kSlotValid = 2u;
constexpr uint32_t kSlotSrcMask = 0xFFFF0u;
constexpr int kSlotDstShift = 20;
inline int64_t fast_slot(int64_t off, int64_t r, int64_t l) { return 64 * off + 256 * (r >> 2) + 4 * l + (r & 3); }

}  // namespace ff
