// Plan: the coefficient support G of Algorithm 1 (steps 3-4), shared by every
// layer that uses the same frames (Sec. 3.3), turned into device index tables
// for the fused kernels, plus the dC workspace.
//
// Canonical coefficient index c = i*rho + 2r + s (subspace i, frame-block r,
// real part s) lives in frame block r at local position 2i + s.  Kernels keep
// one token's coefficients in LDS block by block with block stride W + pad,
// so every table stores LDS element offsets r*(W + pad) + 2i + s directly.
#include <algorithm>
#include <cstring>
#include <functional>
#include <memory>
#include <numeric>

#include "ff_internal.h"

namespace {

struct Loc {
  int blk;
  int local;
};

Loc locate(int64_t c, int64_t rho) {
  const int64_t i = c / rho, rem = c % rho;
  return {(int)(rem / 2), (int)(2 * i + rem % 2)};
}

// Token stride of an LDS tile (elements): whole blocks plus a pad chosen so
// that consecutive token rows start 16 bytes apart modulo 128 bytes, which
// spreads the per-token accesses of the sparse phases over different banks.
int token_stride(int nblk, int ldb, int esz) {
  const int base = nblk * ldb;                 // multiple of 8 elements
  const int period = 128 / esz, want = 16 / esz;
  int pad = ((want - base) % period + period) % period;
  return base + pad;
}

// Byte offset of coefficient `local` of block parity `par` in a 128-wide kernel's pair tile:
// 128 rows of 32 bytes, each holding one coefficient's 8 tokens of both blocks.  Row order
// within 32 coefficients swaps bit 2 of the coefficient with bits 3..4, so that each transposed
// read of the synthesis operand covers 512 contiguous bytes; rows with bit 2 set hold block 1
// first, so that the analysis writes of 16 consecutive coefficients hit distinct LDS banks.
uint32_t tile_byte(int par, int local) {
  const int b2 = (local >> 2) & 1;
  const int row = (local & ~31) | (b2 << 4) | (((local >> 3) & 3) << 2) | (local & 3);
  return (uint32_t)(row * 32 + 16 * (par ^ b2));
}

// Round schedule of the rows of one pair of blocks for the 128-wide kernels.  All 64 lanes of
// a wave run the same rounds, of L[0..R-1] slots; at the end of every round each lane writes
// its current row to the pair tile, so row ends cost no per-slot test.  A row fills one or
// more consecutive rounds of one lane, the rest of its last round being padding slots with
// zero coefficients; a lane whose rows are done rewrites its last row.
struct Span {
  int row, first, last;   // rounds first..last of one lane
};
struct PairSchedule {
  std::vector<int> L;
  std::vector<std::vector<Span>> lanes = std::vector<std::vector<Span>>(64);
};

// Rows (longest first) each to the lane where they end in the earliest round, then with the
// least padding, then the lowest lane; every lane's rounds fill from round 0.  Returns false
// when some row fits on no lane.
bool place_rows(const std::vector<int>& rows, const std::vector<int>& size, const std::vector<int>& L,
                std::vector<std::vector<Span>>* lanes) {
  const int R = (int)L.size();
  std::vector<int> cum(R + 1, 0);
  for (int j = 0; j < R; ++j) cum[j + 1] = cum[j] + L[j];
  // free[f]: lanes whose first free round is f, highest index first
  std::vector<std::vector<int>> free(R + 1);
  for (int l = 63; l >= 0; --l) free[0].push_back(l);
  for (int r : rows) {
    int bb = -1, bw = 0, bf = -1;
    for (int f = 0; f < R; ++f) {
      if (free[f].empty()) continue;
      const int idx = (int)(std::lower_bound(cum.begin(), cum.end(), cum[f] + size[r]) - cum.begin());
      if (idx > R) continue;
      const int b = idx - 1, w = cum[idx] - cum[f] - size[r];
      if (bf < 0 || b < bb || (b == bb && (w < bw || (w == bw && free[f].back() < free[bf].back())))) {
        bb = b;
        bw = w;
        bf = f;
      }
    }
    if (bf < 0) return false;
    const int lane = free[bf].back();
    free[bf].pop_back();
    auto& dst = free[bb + 1];
    dst.insert(std::upper_bound(dst.begin(), dst.end(), lane, std::greater<int>()), lane);
    if (lanes) (*lanes)[lane].push_back({r, bf, bb});
  }
  return true;
}

// Round lengths: the longest row of each group of 64 rows (always placeable), then shortened
// or dropped by local search while the modelled cost falls: `slot_cost` per slot of the
// stream (whole 4-slot groups), `end_cost` per round.
PairSchedule schedule_pair(const std::vector<int>& size, int slot_cost, int end_cost) {
  PairSchedule ps;
  std::vector<int> rows;
  for (int r = 0; r < (int)size.size(); ++r)
    if (size[r] > 0) rows.push_back(r);
  std::stable_sort(rows.begin(), rows.end(), [&](int a, int b) { return size[a] > size[b]; });
  if (rows.empty()) return ps;
  std::vector<int> L;
  for (size_t j = 0; j < rows.size(); j += 64) L.push_back(size[rows[j]]);
  struct Cost {
    int64_t model, sum, rounds;
    bool operator<(const Cost& o) const {
      return model != o.model ? model < o.model : sum != o.sum ? sum < o.sum : rounds < o.rounds;
    }
  };
  auto cost = [&](const std::vector<int>& v) {
    const int64_t sum = std::accumulate(v.begin(), v.end(), (int64_t)0);
    return Cost{slot_cost * std::max<int64_t>((sum + 3) / 4 * 4, 4) + end_cost * (int64_t)v.size(), sum,
                (int64_t)v.size()};
  };
  Cost best = cost(L);
  for (int iter = 0; iter < 4096; ++iter) {
    std::vector<std::vector<int>> cand;
    for (size_t j = 0; j < L.size(); ++j) {
      if (L[j] > 1) {
        std::vector<int> m = L;
        --m[j];
        cand.push_back(m);
        for (int t = 1; t <= 3; ++t) {
          cand.push_back(m);
          cand.back().push_back(t);
        }
      }
      if (L.size() > 1) {
        cand.push_back(L);
        cand.back().erase(cand.back().begin() + (long)j);
      }
    }
    std::stable_sort(cand.begin(), cand.end(),
                     [&](const std::vector<int>& a, const std::vector<int>& b) { return cost(a) < cost(b); });
    bool moved = false;
    for (const auto& m : cand) {
      const Cost c = cost(m);
      if (!(c < best)) break;
      if (place_rows(rows, size, m, nullptr)) {
        L = m;
        best = c;
        moved = true;
        break;
      }
    }
    if (!moved) break;
  }
  ps.L = L;
  place_rows(rows, size, L, &ps.lanes);
  return ps;
}

// Slot words of one pair's stream under its schedule, lane by lane: `entries[r]` are the
// entries of row r, `word(e)` an entry's source-row bits, `dst(r)` row r's tile bits; `put`
// receives (stream row k, lane, word, entry or -1).  Returns the stream length (whole 4-row
// groups, at least one), or -1 if a lane holds no row and the pair has no empty row, and sets
// the round-end mask words.
template <class Word, class Dst, class Put>
int emit_pair(const PairSchedule& ps, const std::vector<std::vector<int>>& entries, Word word, Dst dst, Put put,
              std::vector<uint32_t>& mask) {
  const int R = (int)ps.L.size();
  std::vector<int> cum(R + 1, 0);
  for (int j = 0; j < R; ++j) cum[j + 1] = cum[j] + ps.L[j];
  const int len = std::max((cum[R] + 3) / 4 * 4, 4);
  mask.assign((size_t)(len + 31) / 32 + 1, 0u);
  for (int j = 0; j < R; ++j) mask[(size_t)(cum[j + 1] - 1) / 32] |= 1u << ((cum[j + 1] - 1) % 32);
  auto is_end = [&](int k) { return (mask[(size_t)k / 32] >> (k % 32)) & 1u; };
  int empty_row = -1;   // a row with no entries, for lanes that hold no row
  for (int r = 0; r < (int)entries.size() && empty_row < 0; ++r)
    if (entries[r].empty()) empty_row = r;
  for (int l = 0; l < 64; ++l) {
    const auto& sp = ps.lanes[l];
    if (sp.empty()) {
      if (empty_row < 0) return -1;
      for (int k = 0; k < len; ++k) put(k, l, is_end(k) ? dst(empty_row) : 0u, -1);
      continue;
    }
    int k = 0;
    for (size_t j = 0; j < sp.size(); ++j) {
      const Span& s = sp[j];
      const int stop = cum[s.last + 1];
      const auto& ent = entries[s.row];
      // the last row is not restarted: the lane's later round ends write it again
      const uint32_t restart = j + 1 < sp.size() ? ff::kSlotEnd : 0u;
      for (; k < stop; ++k) {
        const int i = k - cum[s.first];
        const bool has = i < (int)ent.size();
        // padding slots name the row only where a round ends (elsewhere their reads all go to
        // offset 0, one LDS broadcast)
        put(k, l,
            has ? word(ent[i]) | ff::kSlotValid | dst(s.row) | (k == stop - 1 ? restart : 0u)
                : (is_end(k) ? dst(s.row) | (k == stop - 1 ? restart : 0u) : 0u),
            has ? ent[i] : -1);
      }
    }
    for (; k < len; ++k) put(k, l, is_end(k) ? dst(sp.back().row) : 0u, -1);   // rewrites of the last row
  }
  return len;
}

}  // namespace

// A generic stream (GenStream) on the host: entry words, the user entry of every stream element
// (-1: padding) and the first row of each wave.
struct StreamHost {
  std::vector<int2> ent;
  std::vector<int> id;
  std::vector<int> wave_row;
  int64_t rows = 0;
};

// Slots are the indices of `lists` (entries of each slot, in stream order), sorted by entry count
// with the longest first; src(e) is the LDS offset an entry reads, dst(slot) where its slot's
// result goes.
template <class Src, class Dst>
StreamHost build_stream(const std::vector<std::vector<int>>& lists, Src src, Dst dst) {
  const int64_t nslots = (int64_t)lists.size(), nslab = (nslots + 63) / 64;
  std::vector<int> order((size_t)nslots);
  std::iota(order.begin(), order.end(), 0);
  std::stable_sort(order.begin(), order.end(), [&](int a, int b) { return lists[a].size() > lists[b].size(); });
  std::vector<int64_t> slab_row((size_t)nslab + 1, 0);
  for (int64_t s = 0; s < nslab; ++s) {
    size_t len = 1;   // every slab has a row, so every slot's result is written
    for (int64_t l = 0; l < 64 && 64 * s + l < nslots; ++l) len = std::max(len, lists[order[64 * s + l]].size());
    slab_row[s + 1] = slab_row[s] + (int64_t)len;
  }
  StreamHost h;
  h.rows = slab_row[nslab];
  h.ent.assign((size_t)(h.rows * 64), make_int2(0, -1));
  h.id.assign((size_t)(h.rows * 64), -1);
  for (int64_t s = 0; s < nslab; ++s) {
    const int64_t len = slab_row[s + 1] - slab_row[s];
    for (int64_t l = 0; l < 64; ++l) {
      const int64_t slot = 64 * s + l;
      const bool real = slot < nslots;
      const int d = real ? dst(order[slot]) : -1;
      for (int64_t k = 0; k < len; ++k) {
        const size_t j = (size_t)((slab_row[s] + k) * 64 + l);
        const int e = real && k < (int64_t)lists[order[slot]].size() ? lists[order[slot]][k] : -1;
        h.ent[j] = make_int2((e >= 0 ? src(e) : 0) | (k == len - 1 ? ff::kRowLast : 0), d);
        h.id[j] = e;
      }
    }
  }
  // waves take contiguous runs of slabs with about equal numbers of rows
  h.wave_row.assign(ff::kGenWaves + 1, (int)h.rows);
  h.wave_row[0] = 0;
  int64_t s = 0;
  for (int w = 1; w < ff::kGenWaves; ++w) {
    const int64_t target = h.rows * w / ff::kGenWaves;
    while (s < nslab && slab_row[s] < target) ++s;
    h.wave_row[w] = (int)std::max<int64_t>(slab_row[s], h.wave_row[w - 1]);
  }
  return h;
}

// Chunk streams are concatenated; each keeps its own wave runs (rows offset by those before).
void append_stream(StreamHost& all, const StreamHost& h) {
  for (int w = 0; w <= ff::kGenWaves; ++w) all.wave_row.push_back((int)(all.rows + h.wave_row[w]));
  all.ent.insert(all.ent.end(), h.ent.begin(), h.ent.end());
  all.id.insert(all.id.end(), h.id.begin(), h.id.end());
  all.rows += h.rows;
}

extern "C" ff_status ff_plan_create(const ff_frame* f_in, const ff_frame* f_out, int64_t nnz,
                                    const int32_t* rows, const int32_t* cols, int64_t max_tokens,
                                    int64_t max_batch, ff_plan** out) {
  ff::clear_error();
  if (!out) return ff::fail(FF_EINVAL, "out is NULL");
  *out = nullptr;
  if (!f_in || !f_out) return ff::fail(FF_EINVAL, "frame is NULL");
  if (f_in->device != f_out->device) return ff::fail(FF_EINVAL, "frames live on different devices");
  const int64_t n = f_in->dv, m = f_out->dv;        // the coefficient grid, (k rho_m) x (k rho_n)
  if (nnz < 0 || nnz > m * n || nnz > ((int64_t)1 << 30))
    return ff::fail(FF_EINVAL, "nnz=%lld out of range", (long long)nnz);
  if (nnz > 0 && (!rows || !cols)) return ff::fail(FF_EINVAL, "rows/cols is NULL");
  if (max_tokens < 0 || max_tokens > ((int64_t)1 << 31) - 1)
    return ff::fail(FF_EINVAL, "max_tokens=%lld out of range", (long long)max_tokens);
  if (max_batch < 1 || max_batch > 65535)
    return ff::fail(FF_EINVAL, "max_batch=%lld out of range", (long long)max_batch);
  for (int64_t e = 0; e < nnz; ++e)
    if (rows[e] < 0 || rows[e] >= m || cols[e] < 0 || cols[e] >= n)
      return ff::fail(FF_EINVAL, "support entry %lld = (%d, %d) outside %lld x %lld", (long long)e,
                      rows[e], cols[e], (long long)m, (long long)n);
  {
    std::vector<int64_t> key((size_t)nnz);
    for (int64_t e = 0; e < nnz; ++e) key[e] = (int64_t)rows[e] * n + cols[e];
    std::sort(key.begin(), key.end());
    for (int64_t e = 1; e < nnz; ++e)
      if (key[e] == key[e - 1])
        return ff::fail(FF_EINVAL, "duplicate support entry (%lld, %lld)", (long long)(key[e] / n),
                        (long long)(key[e] % n));
  }

  const ff::FrameDev& FI = f_in->dev;
  const ff::FrameDev& FO = f_out->dev;
  std::unique_ptr<ff_plan> p(new ff_plan());
  p->fin = const_cast<ff_frame*>(f_in);
  p->fout = const_cast<ff_frame*>(f_out);
  p->nnz = nnz;
  p->max_tokens = max_tokens;
  p->max_batch = max_batch;
  p->device = f_in->device;
  p->ldb_in = ff::lds_block_span(FI) + ff::kBlockPad;
  p->ldb_out = ff::lds_block_span(FO) + ff::kBlockPad;
  for (int dt = 0; dt < 2; ++dt) {
    const int esz = dt == FF_BF16 ? 2 : 4;
    p->ldt_in[dt] = token_stride(FI.nblk, p->ldb_in, esz);
    p->ldt_out[dt] = token_stride(FO.nblk, p->ldb_out, esz);
    const int64_t per_token = (int64_t)(p->ldt_in[dt] + p->ldt_out[dt]) * esz;
    int64_t tt = (ff::kMaxLdsBytes - ff::kTwLdsBytes) / per_token;
    if (tt < 1)
      return ff::fail(FF_EUNSUPPORTED, "one token of %lld + %lld coefficients exceeds LDS", (long long)n,
                      (long long)m);
    tt = std::min<int64_t>(tt, ff::kMaxTileTokens);
    p->tile_tokens[dt] = (int)tt;
    p->lds_bytes[dt] = (size_t)(tt * per_token) + ff::kTwLdsBytes;
  }
  // Generic kernels: the output side (v in the forward, u in the backward) is needed whole, but
  // the input side (z, q) only one chunk of input blocks at a time, so chunking lets a tile hold
  // more tokens (fewer passes over the stream tables and, backward, fewer dC partial-row updates
  // per token, at the price of a barrier-separated phase sequence per chunk).  It pays where the
  // stream dominates, nnz >= 4 (n + m) (measured on the backward: the 70B down projection 25%
  // faster; the 7B MLP down projection about even at 50k coefficients and 9% slower at 10k).
  // The chunk count is the smallest one that reaches min(8, twice the whole-tile count) tokens
  // in bf16 (the same chunks serve fp32), else 1.
  auto chunk_tokens = [&](int nch, int dt) -> int64_t {
    const int esz = dt == FF_BF16 ? 2 : 4;
    const int ldc = token_stride((FI.nblk + nch - 1) / nch, p->ldb_in, esz);
    const int64_t tt = (ff::kMaxLdsBytes - ff::kTwLdsBytes) / ((int64_t)(p->ldt_out[dt] + ldc) * esz);
    return std::min<int64_t>(tt, ff::kMaxTileTokens);
  };
  {
    const int64_t whole = chunk_tokens(1, FF_BF16), want = std::min<int64_t>(8, 2 * whole);
    int nch = 1;
    const bool dense_stream = nnz >= 4 * (n + m);
    for (int c = 2; dense_stream && whole < want && c <= std::min(FI.nblk, ff::kMaxGenChunks); ++c)
      if (chunk_tokens(c, FF_BF16) >= want) {
        nch = c;
        break;
      }
    p->gen_nch = nch;
    for (int c = 0; c <= nch; ++c) p->gen_chunk_blk[c] = (int)((int64_t)c * FI.nblk / nch);
    // bf16 token-grouped tiles (gen_kernels.h): every table row of the sparse phases reads four
    // tokens per LDS access; they need whole groups of four tokens, and frames whose blocks are
    // applied directly (up to 128 wide) or in one radix-4 stage
    auto grouped_ok = [](const ff::FrameDev& f) {
      return (f.radix == 1 && f.nst == 0 && f.W <= 128) || (f.radix == 4 && f.nst == 1 && f.W2 <= 128);
    };
    p->gen_g4 = grouped_ok(FI) && grouped_ok(FO) && !f_in->lifted && !f_out->lifted && chunk_tokens(nch, FF_BF16) >= 4;
    for (int dt = 0; dt < 2; ++dt) {
      const int esz = dt == FF_BF16 ? 2 : 4;
      p->gen_ldt_in[dt] = token_stride((FI.nblk + nch - 1) / nch, p->ldb_in, esz);
      p->gen_tile_tokens[dt] = (int)chunk_tokens(nch, dt);
      if (dt == FF_BF16 && p->gen_g4) p->gen_tile_tokens[dt] &= ~3;
      p->gen_lds_bytes[dt] = (size_t)p->gen_tile_tokens[dt] * (size_t)(p->ldt_out[dt] + p->gen_ldt_in[dt]) * esz +
                             ff::kTwLdsBytes;
    }
  }

  // ---------------- host tables
  std::vector<Loc> rloc((size_t)nnz), cloc((size_t)nnz);
  for (int64_t e = 0; e < nnz; ++e) {
    rloc[e] = locate(rows[e], f_out->rho);
    cloc[e] = locate(cols[e], f_in->rho);
  }
  auto off_out = [&](const Loc& l) { return l.blk * p->ldb_out + ff::lds_position(FO, l.local); };
  auto off_in = [&](const Loc& l) { return l.blk * p->ldb_in + ff::lds_position(FI, l.local); };

  // generic streams: v = C z over the rows of C and q = C^T u over its columns, slots sorted
  // by entry count (longest first), entries within a slot in order of their other index
  std::vector<std::vector<int>> by_row((size_t)m), by_col((size_t)n);
  {
    std::vector<int64_t> byc((size_t)nnz), byr((size_t)nnz);
    std::iota(byc.begin(), byc.end(), 0);
    std::iota(byr.begin(), byr.end(), 0);
    std::stable_sort(byc.begin(), byc.end(), [&](int64_t a, int64_t b) { return cols[a] < cols[b]; });
    std::stable_sort(byr.begin(), byr.end(), [&](int64_t a, int64_t b) { return rows[a] < rows[b]; });
    for (int64_t e : byc) by_row[rows[e]].push_back((int)e);
    for (int64_t e : byr) by_col[cols[e]].push_back((int)e);
  }
  // the forward stream: one stream per input-side chunk over every row of C (the row's entries
  // in that chunk; sources relative to the chunk's first block), concatenated
  StreamHost gfwd;
  for (int ch = 0; ch < p->gen_nch; ++ch) {
    const int b0 = p->gen_chunk_blk[ch], b1 = p->gen_chunk_blk[ch + 1];
    std::vector<std::vector<int>> lists((size_t)m);
    for (int64_t r = 0; r < m; ++r)
      for (int e : by_row[r])
        if (cloc[e].blk >= b0 && cloc[e].blk < b1) lists[r].push_back(e);
    const StreamHost h = build_stream(
        lists, [&](int e) { return off_in(Loc{cloc[e].blk - b0, cloc[e].local}); },
        [&](int64_t r) { return off_out(locate(r, f_out->rho)); });
    append_stream(gfwd, h);
  }
  // the backward stream: one stream per input-side chunk (its columns, destinations relative to
  // the chunk's first block), concatenated, with per-chunk wave runs
  StreamHost gbwd;
  for (int ch = 0; ch < p->gen_nch; ++ch) {
    const int b0 = p->gen_chunk_blk[ch], b1 = p->gen_chunk_blk[ch + 1];
    std::vector<int64_t> col_of;
    std::vector<std::vector<int>> lists;
    for (int64_t c = 0; c < n; ++c) {
      const int blk = locate(c, f_in->rho).blk;
      if (blk >= b0 && blk < b1) {
        col_of.push_back(c);
        lists.push_back(by_col[c]);
      }
    }
    const StreamHost h = build_stream(
        lists, [&](int e) { return off_out(rloc[e]); },
        [&](int64_t slot) {
          const Loc l = locate(col_of[slot], f_in->rho);
          return off_in(Loc{l.blk - b0, l.local});
        });
    append_stream(gbwd, h);
  }
  {
    // every stream offset stays inside its tile row (output side whole, input side one chunk)
    const int cmax = (FI.nblk + p->gen_nch - 1) / p->gen_nch;
    for (const int2& e : gbwd.ent) {
      const int so = e.x & ~ff::kRowLast;
      if (so < 0 || so >= FO.nblk * p->ldb_out || e.y < -1 || e.y >= cmax * p->ldb_in)
        return ff::fail(FF_EINVAL, "internal: backward stream offset outside its tile");
    }
    for (const int2& e : gfwd.ent) {
      const int so = e.x & ~ff::kRowLast;
      if (so < 0 || so >= cmax * p->ldb_in || e.y < -1 || e.y >= FO.nblk * p->ldb_out)
        return ff::fail(FF_EINVAL, "internal: forward stream offset outside its tile");
    }
  }
  // merge buckets (R, S)
  const int64_t nb = (int64_t)FO.nblk * FI.nblk;
  std::vector<int> mrg_ptr((size_t)nb + 1, 0);
  for (int64_t e = 0; e < nnz; ++e) mrg_ptr[(int64_t)rloc[e].blk * FI.nblk + cloc[e].blk + 1]++;
  int max_bucket = 0;
  for (int64_t b = 0; b < nb; ++b) {
    max_bucket = std::max(max_bucket, mrg_ptr[b + 1]);
    mrg_ptr[b + 1] += mrg_ptr[b];
  }
  std::vector<int4> mrg_ent((size_t)std::max<int64_t>(nnz, 1));
  {
    std::vector<int> pos(mrg_ptr.begin(), mrg_ptr.end() - 1);
    for (int64_t e = 0; e < nnz; ++e) {
      const int64_t b = (int64_t)rloc[e].blk * FI.nblk + cloc[e].blk;
      mrg_ent[pos[b]++] = make_int4(rloc[e].local, cloc[e].local, (int)e, 0);
    }
  }

  // ---------------- 128-wide fused path: balanced entry streams per pair of blocks
  // Forward stream (v = C z), one per pair of output blocks, slot words as described with
  // kSlotEnd in ff_internal.h.  The plan's coefficient layout is this stream's slot layout, so
  // forward slots read coefficients without an index; slots that hold no entry are padding.
  // Backward stream (dC and q = C^T u), one per pair of input blocks, grouped by column
  // of C: (byte offset of the source row of u | tile row of the column | end-of-column | valid,
  // coefficient slot).
  const bool fast = !f_in->lifted && !f_out->lifted && FI.W == 128 && FO.W == 128 && FI.nblk % 2 == 0 &&
                    FO.nblk % 2 == 0 &&
                    f_in->transpose_is_sign_flip && f_in->half_shift_sign && f_in->B == f_out->B &&
                    n < 65536 && m < 65536 &&
                    ff::fast128_lds_bytes(std::max(FI.nblk, FO.nblk)) <= (size_t)ff::kMaxLdsBytes;
  std::vector<int4> f_pl, b_pl;   // per pair: (first stream row, stream rows, mask offset, mask word 0)
  std::vector<uint32_t> f_em, b_em;   // round-end masks
  std::vector<int> pad_slots;
  std::vector<uint32_t> f_st;
  std::vector<uint2> b_st;
  std::vector<int> slot_of_user((size_t)nnz), bwd_slot_of_user;
  std::vector<int64_t> user_of_slot;
  bool bwd16 = false;
  if (fast) {
    // byte offset of a coefficient's row in the LDS array of a whole side, and its row in a pair tile
    auto lsrc = [&](const Loc& l) { return (uint32_t)(l.blk * 128 + l.local) * 16u; };
    const int npo = FO.nblk / 2, npi = FI.nblk / 2;
    // entries of each destination row r = (block parity)*128 + local of a pair
    std::vector<std::vector<std::vector<int>>> frows(npo, std::vector<std::vector<int>>(256)),
        brows(npi, std::vector<std::vector<int>>(256));
    for (int64_t e = 0; e < nnz; ++e) {
      frows[rloc[e].blk / 2][(rloc[e].blk & 1) * 128 + rloc[e].local].push_back((int)e);
      brows[cloc[e].blk / 2][(cloc[e].blk & 1) * 128 + cloc[e].local].push_back((int)e);
    }
    // modelled VALU work per slot and per round end of the two kernels' sparse phases
    constexpr int kFwdSlotCost = 11, kBwdSlotCost = 17, kEndCost = 15;
    std::vector<uint32_t> mask;
    for (int pp = 0; pp < npo; ++pp) {
      std::vector<int> sz(256);
      for (int r = 0; r < 256; ++r) sz[r] = (int)frows[pp][r].size();
      const PairSchedule ps = schedule_pair(sz, kFwdSlotCost, kEndCost);
      const size_t row0 = f_st.size() / 64;
      // at most 64 x 256 x 2^15 slots per stream keep every offset in an int
      const int len = emit_pair(
          ps, frows[pp], [&](int e) { return lsrc(cloc[e]); },
          [&](int r) { return tile_byte(r >> 7, r & 127) << ff::kSlotDstShift; },
          [&](int k, int l, uint32_t w, int e) {
            const size_t slot = (size_t)ff::fast_slot((int64_t)row0, k, l);
            if (slot >= f_st.size()) {
              f_st.resize(slot / 256 * 256 + 256, 0u);
              user_of_slot.resize(f_st.size(), -1);
            }
            f_st[slot] = w;
            if (e >= 0) {
              user_of_slot[slot] = e;
              slot_of_user[e] = (int)slot;
            }
          },
          mask);
      if (len < 0) return ff::fail(FF_EUNSUPPORTED, "internal: no row for a lane of output pair %d", pp);
      f_pl.push_back(make_int4((int)row0, len, (int)f_em.size(), (int)mask[0]));
      f_em.insert(f_em.end(), mask.begin(), mask.end());
      f_st.resize((row0 + (size_t)len) * 64, 0u);
      user_of_slot.resize(f_st.size(), -1);
    }
    for (size_t j = 0; j < user_of_slot.size(); ++j)
      if (user_of_slot[j] < 0) pad_slots.push_back((int)j);
    bwd_slot_of_user.assign((size_t)nnz, 0);
    for (int pp = 0; pp < npi; ++pp) {
      std::vector<int> sz(256);
      for (int r = 0; r < 256; ++r) sz[r] = (int)brows[pp][r].size();
      const PairSchedule ps = schedule_pair(sz, kBwdSlotCost, kEndCost);
      const int64_t row0 = (int64_t)(b_st.size() / 64);
      const int len = emit_pair(
          ps, brows[pp], [&](int e) { return lsrc(rloc[e]); },
          [&](int r) { return tile_byte(r >> 7, r & 127) << ff::kSlotDstShift; },
          [&](int k, int l, uint32_t w, int e) {
            const size_t slot = (size_t)ff::fast_slot(row0, k, l);
            if (slot >= b_st.size()) b_st.resize(slot / 256 * 256 + 256, make_uint2(0u, 0u));
            b_st[slot] = make_uint2(w, e >= 0 ? (unsigned)slot_of_user[e] : 0u);
            if (e >= 0) bwd_slot_of_user[e] = (int)slot;
          },
          mask);
      if (len < 0) return ff::fail(FF_EUNSUPPORTED, "internal: no row for a lane of input pair %d", pp);
      b_pl.push_back(make_int4((int)row0, len, (int)b_em.size(), (int)mask[0]));
      b_em.insert(b_em.end(), mask.begin(), mask.end());
      b_st.resize((size_t)(row0 + len) * 64, make_uint2(0u, 0u));
    }
    // The 16-token backward holds a whole stream in registers and the output side's array for
    // 16 tokens in LDS; its slot words address rows of 32 bytes instead of 16, at the row's
    // first token half, which row c keeps at bytes 16 (c & 1).
    int max_len = 0;
    for (const int4& e : b_pl) max_len = std::max(max_len, e.y);
    bwd16 = max_len <= 16 && ff::fast16_lds_bytes(FO.nblk) <= (size_t)ff::kMaxLdsBytes;
    if (bwd16)
      for (uint2& w : b_st) {
        const uint32_t row = (w.x & ff::kSlotSrcMask) >> 4;
        w.x = (w.x & ~ff::kSlotSrcMask) | (row * 32 + 16 * (row & 1));
      }
  } else {
    // the generic kernels' layout is the forward stream's entry order, padding included, so
    // the forward reads coefficients by stream position
    user_of_slot.assign(gfwd.id.begin(), gfwd.id.end());
    for (size_t j = 0; j < gfwd.id.size(); ++j)
      if (gfwd.id[j] >= 0) slot_of_user[gfwd.id[j]] = (int)j;
  }
  const int64_t nslot = (int64_t)user_of_slot.size();   // coefficient slots (>= nnz)
  // for the 128-wide backward: the backward slot of every coefficient slot (padding slots go
  // to the scratch slot just past the backward slots)
  std::vector<int> bwd_pos;
  if (fast) {
    bwd_pos.resize((size_t)nslot);
    for (int64_t j = 0; j < nslot; ++j)
      bwd_pos[j] = user_of_slot[j] >= 0 ? bwd_slot_of_user[user_of_slot[j]] : (int)b_st.size();
  }
  for (auto& en : mrg_ent) en.z = nnz ? slot_of_user[en.z] : 0;
  // coefficient slot of every generic stream element (-1: padding), and the slots with no entry
  std::vector<int> fcoef(gfwd.id.size()), bcoef(gbwd.id.size()), coef_pad;
  for (size_t j = 0; j < fcoef.size(); ++j) fcoef[j] = gfwd.id[j] >= 0 ? slot_of_user[gfwd.id[j]] : -1;
  for (size_t j = 0; j < bcoef.size(); ++j) bcoef[j] = gbwd.id[j] >= 0 ? slot_of_user[gbwd.id[j]] : -1;
  for (int64_t j = 0; j < nslot; ++j)
    if (user_of_slot[j] < 0) coef_pad.push_back((int)j);
  const size_t gf_elems = gfwd.ent.size(), gb_elems = gbwd.ent.size();
  p->user_order = std::move(user_of_slot);
  p->coef_slots = nslot;
  const int64_t fast_tiles = fast ? (max_tokens + ff::kFastTileTokens - 1) / ff::kFastTileTokens : 0;
  // the backward stream as the kernel's slot words and the reduction's destinations
  std::vector<uint32_t> b_w(b_st.size()), b_dst(b_st.size());
  std::vector<int> b_pad;   // backward slots that hold no entry (zero coefficients in any copy)
  for (size_t i = 0; i < b_st.size(); ++i) {
    b_w[i] = b_st[i].x;
    b_dst[i] = (b_st[i].x & ff::kSlotValid) ? b_st[i].y : ~0u;
    if (!(b_st[i].x & ff::kSlotValid)) b_pad.push_back((int)i);
  }
  if (b_pad.empty()) b_pad.push_back((int)b_st.size());   // the copy's scratch slot stands in

  // ---------------- device memory: one allocation for every table and the workspace
  auto up = [](size_t x) { return (x + 255) & ~(size_t)255; };
  // the generic backward runs at most one workgroup per CU and adapter, each accumulating the
  // dC partial sums of all its tiles in one row
  {
    int ncu = 0;
    if (hipDeviceGetAttribute(&ncu, hipDeviceAttributeMultiprocessorCount, p->device) != hipSuccess || ncu < 1)
      return ff::fail(FF_EDEVICE, "querying the device's compute units failed");
    p->gen_wgs = ncu;
  }
  // (a call may use tiles of fewer tokens than the LDS allows, so up to one tile per token)
  p->gen_rows = (int)std::max<int64_t>(1, std::min<int64_t>(max_tokens, p->gen_wgs));
  const size_t partial_elems = std::max((size_t)max_batch * (size_t)p->gen_rows * gb_elems,
                                        (size_t)max_batch * (size_t)fast_tiles *
                                            (fast ? ff::fast128_partial_floats(b_st.size()) : 0));
  struct Blob {
    const void* src;
    size_t bytes;
  };
  enum {
    kGfEnt, kGfCoef, kGfWave, kGbEnt, kGbCoef, kGbWave, kCoefPad, kCfwd, kCbwd, kMrgPtr, kMrgEnt,
    kFPl, kBPl, kFSt, kPadSlots, kBW, kPartial, kCoefBwd, kBwdPos, kFEm, kBDst, kBEm, kBPad, kUserOfSlot,
    kSlotOfUser, kMrgG, kMrgOut, kLiftX, kLiftG, kLiftDX, kNumBlobs
  };
  // frames with a lift merge through the backward, a chunk of (user) rows at a time
  const bool lifted = f_in->lifted || f_out->lifted;
  const bool mrg_transform = lifted;
  const int64_t mrg_rows = mrg_transform ? std::min<int64_t>(f_out->d, 1024) : 0;
  const size_t lift_rows = lifted ? (size_t)max_tokens : 0;
  // both directions of the coefficient layout, for the device-side conversions
  std::vector<int> user_of_slot32(p->user_order.begin(), p->user_order.end());
  std::vector<Blob> blobs(kNumBlobs);
  blobs[kGfEnt] = {gfwd.ent.data(), gf_elems * sizeof(int2)};
  blobs[kGfCoef] = {fcoef.data(), gf_elems * sizeof(int)};
  blobs[kGfWave] = {gfwd.wave_row.data(), gfwd.wave_row.size() * sizeof(int)};
  blobs[kGbEnt] = {gbwd.ent.data(), gb_elems * sizeof(int2)};
  blobs[kGbCoef] = {bcoef.data(), gb_elems * sizeof(int)};
  blobs[kGbWave] = {gbwd.wave_row.data(), gbwd.wave_row.size() * sizeof(int)};
  blobs[kCoefPad] = {coef_pad.data(), coef_pad.size() * sizeof(int)};
  // per-call coefficient copies in the generic streams' orders (the forward's only when the
  // coefficient layout is not already its order)
  blobs[kCfwd] = {nullptr, (fast ? (size_t)max_batch * gf_elems : 1) * sizeof(float)};
  blobs[kCbwd] = {nullptr, (size_t)max_batch * gb_elems * sizeof(float)};
  blobs[kMrgPtr] = {mrg_ptr.data(), (nb + 1) * sizeof(int)};
  blobs[kMrgEnt] = {mrg_ent.data(), mrg_ent.size() * sizeof(int4)};
  blobs[kFPl] = {f_pl.data(), f_pl.size() * sizeof(int4)};
  blobs[kBPl] = {b_pl.data(), b_pl.size() * sizeof(int4)};
  blobs[kFSt] = {f_st.data(), f_st.size() * sizeof(uint32_t)};
  blobs[kPadSlots] = {pad_slots.data(), pad_slots.size() * sizeof(int)};
  blobs[kBW] = {b_w.data(), b_w.size() * sizeof(uint32_t)};
  blobs[kPartial] = {nullptr, std::max<size_t>(partial_elems, 1) * sizeof(float)};
  // the backward's coefficients in its stream's slot order, per adapter (+ a scratch group)
  blobs[kCoefBwd] = {nullptr, std::max<size_t>((size_t)max_batch * (b_st.size() + 256), 1) * sizeof(float)};
  blobs[kBwdPos] = {bwd_pos.data(), bwd_pos.size() * sizeof(int)};
  blobs[kFEm] = {f_em.data(), f_em.size() * sizeof(uint32_t)};
  blobs[kBDst] = {b_dst.data(), b_dst.size() * sizeof(uint32_t)};
  blobs[kBEm] = {b_em.data(), b_em.size() * sizeof(uint32_t)};
  blobs[kBPad] = {b_pad.data(), b_pad.size() * sizeof(int)};
  blobs[kUserOfSlot] = {user_of_slot32.data(), user_of_slot32.size() * sizeof(int)};
  blobs[kSlotOfUser] = {slot_of_user.data(), (size_t)nnz * sizeof(int)};
  blobs[kMrgG] = {nullptr, (size_t)mrg_rows * (size_t)m * sizeof(float)};
  blobs[kMrgOut] = {nullptr, (size_t)mrg_rows * (size_t)n * sizeof(float)};
  blobs[kLiftX] = {nullptr, lift_rows * (size_t)n * sizeof(float)};
  blobs[kLiftG] = {nullptr, lift_rows * (size_t)m * sizeof(float)};
  blobs[kLiftDX] = {nullptr, lift_rows * (size_t)n * sizeof(float)};
  size_t total = 0;
  for (const Blob& b : blobs) total += up(b.bytes);
  int cur = 0;
  if (hipGetDevice(&cur) != hipSuccess || cur != p->device)
    return ff::fail(FF_EDEVICE, "current device differs from the frames' device");
  void* mem = nullptr;
  if (hipMalloc(&mem, total) != hipSuccess) {
    (void)hipGetLastError();
    return ff::fail(FF_ENOMEM, "hipMalloc of %zu bytes for the plan failed", total);
  }
  std::vector<void*> where;
  {
    size_t off = 0;
    for (const Blob& b : blobs) {
      void* dst = (char*)mem + off;
      off += up(b.bytes);
      if (b.src && b.bytes && hipMemcpy(dst, b.src, b.bytes, hipMemcpyHostToDevice) != hipSuccess) {
        (void)hipFree(mem);
        return ff::fail(FF_EDEVICE, "copying plan tables to the device failed");
      }
      where.push_back(dst);
    }
  }
  // the backward's padding slots keep zero coefficients: the per-call copy writes only the
  // slots that hold entries
  if (hipMemset(where[kCoefBwd], 0, blobs[kCoefBwd].bytes) != hipSuccess) {
    (void)hipFree(mem);
    return ff::fail(FF_EDEVICE, "clearing the plan workspace failed");
  }
  ff::PlanDev& pd = p->dev;
  pd.fwd = {(const int2*)where[kGfEnt], (const int*)where[kGfCoef], (const int*)where[kGfWave], (int)gfwd.rows};
  pd.bwd = {(const int2*)where[kGbEnt], (const int*)where[kGbCoef], (const int*)where[kGbWave], (int)gbwd.rows};
  pd.fwd_by_pos = fast ? 0 : 1;
  pd.coef_pad = (const int*)where[kCoefPad];
  pd.ncoef_pad = (int)coef_pad.size();
  pd.c_fwd = (float*)where[kCfwd];
  pd.c_bwd = (float*)where[kCbwd];
  pd.mrg_ptr = (const int*)where[kMrgPtr];
  pd.mrg_ent = (const int4*)where[kMrgEnt];
  pd.mrg_max_bucket = max_bucket;
  pd.nnz = (int)nslot;
  pd.user_of_slot = (const int*)where[kUserOfSlot];
  pd.slot_of_user = (const int*)where[kSlotOfUser];
  pd.nnz_user = (int)nnz;
  p->mrg_rows = (int)mrg_rows;
  p->mrg_g = (float*)where[kMrgG];
  p->mrg_out = (float*)where[kMrgOut];
  p->lifted = lifted;
  p->lift_x = (float*)where[kLiftX];
  p->lift_g = (float*)where[kLiftG];
  p->lift_dx = (float*)where[kLiftDX];
  ff::FastPlanDev& fp = p->fast;
  fp.enabled = fast ? 1 : 0;
  fp.fwd_pl = (const int4*)where[kFPl];
  fp.bwd_pl = (const int4*)where[kBPl];
  fp.fwd_em = (const uint32_t*)where[kFEm];
  fp.fwd_st = (const uint32_t*)where[kFSt];
  fp.pad = (const int*)where[kPadSlots];
  fp.npad = (int)pad_slots.size();
  fp.bwd_st = (const uint32_t*)where[kBW];
  fp.bwd_dst = (const uint32_t*)where[kBDst];
  fp.bwd_em = (const uint32_t*)where[kBEm];
  fp.bwd_pad = (const int*)where[kBPad];
  fp.nbpad = (int)b_pad.size();
  fp.bwd_slots = (int)b_st.size();
  p->partial = (float*)where[kPartial];
  fp.coef_bwd = (float*)where[kCoefBwd];
  fp.bwd_pos = (const int*)where[kBwdPos];
  fp.coef_slots = (int)nslot;
  fp.bwd16 = bwd16 ? 1 : 0;
  p->dev_mem = mem;
  p->workspace_bytes = total;
  p->fin->refs.fetch_add(1);
  p->fout->refs.fetch_add(1);
  *out = p.release();
  return FF_OK;
}

extern "C" void ff_plan_destroy(ff_plan* p) {
  if (!p) return;
  if (p->dev_mem) (void)hipFree(p->dev_mem);
  ff_frame_destroy(p->fin);
  ff_frame_destroy(p->fout);
  delete p;
}

extern "C" ff_status ff_plan_order(const ff_plan* p, int64_t* user_index) {
  ff::clear_error();
  if (!p || (!user_index && p->coef_slots > 0)) return ff::fail(FF_EINVAL, "NULL argument");
  for (int64_t j = 0; j < p->coef_slots; ++j) user_index[j] = p->user_order[j];
  return FF_OK;
}

extern "C" ff_status ff_plan_query(const ff_plan* p, int key, int64_t* value) {
  ff::clear_error();
  if (!p || !value) return ff::fail(FF_EINVAL, "NULL argument");
  switch (key) {
    case FF_Q_TOKENS_PER_TILE_F32: *value = p->tile_tokens[FF_F32]; return FF_OK;
    case FF_Q_TOKENS_PER_TILE_BF16: *value = p->tile_tokens[FF_BF16]; return FF_OK;
    case FF_Q_WORKSPACE_BYTES: *value = (int64_t)p->workspace_bytes; return FF_OK;
    case FF_Q_NNZ: *value = p->nnz; return FF_OK;
    case FF_Q_FAST128: *value = p->fast.enabled; return FF_OK;
    case FF_Q_COEF_SLOTS: *value = p->coef_slots; return FF_OK;
    case FF_Q_SAVED_FLOATS: *value = p->fast.enabled ? (int64_t)p->fast.bwd_slots + 256 : 0; return FF_OK;
    case FF_Q_BWD_TILE_TOKENS: *value = !p->fast.enabled ? 0 : p->fast.bwd16 ? 16 : 8; return FF_OK;
    case FF_Q_RADIX_IN: *value = p->fin->dev.radix; return FF_OK;
    case FF_Q_RADIX_OUT: *value = p->fout->dev.radix; return FF_OK;
    case FF_Q_GEN_CHUNKS: *value = p->gen_nch; return FF_OK;
    case FF_Q_GEN_TILE_TOKENS_F32: *value = p->gen_tile_tokens[FF_F32]; return FF_OK;
    case FF_Q_GEN_TILE_TOKENS_BF16: *value = p->gen_tile_tokens[FF_BF16]; return FF_OK;
    case FF_Q_GEN_TOKEN_GROUPS: *value = p->gen_g4; return FF_OK;
    default: return ff::fail(FF_EINVAL, "unknown query key %d", key);
  }
}
