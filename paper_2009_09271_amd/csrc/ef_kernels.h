// HIP kernels of the efsparse hot path (gfx950).
//
// The plain streaming kernels give each thread one coalesced float4 group (64-thread workgroups,
// kRbTile elements each).  The selection kernels work on rows: a row is the part of one segment
// inside one data tile of kTile elements, so that every workgroup of the selection pipeline serves
// exactly one segment.
//
// Top-k and random-k (Section 3) share one pipeline; no kernel synchronises across workgroups:
//   k_sample_gather  top-k only: the keys of a sample per segment (the whole segment when it has
//   k_sample_select  at most kExactMax elements, else runs spread over it); per segment either
//                    the exact winner rule (small segments) or a candidate threshold set so that
//                    the candidates very likely number at least k_l.
//   k_stream_sel     per row: fused accumulate (acc = g + e, written to e), candidate test (top-k:
//                    the rule above; random-k: Philox key < tau_l, a binomial bound on k_l), the
//                    row's candidates in index order to its slot, and a histogram of them (top-k).
//                    Random-k on layouts whose rows and key window fit k_select's LDS: also the
//                    row's certain winners (key < ulo_l) counted and its undecided candidates
//                    listed, so that k_collect is not needed.
//   k_resolve        top-k, per segment: the histogram bin holding the k_l-th best candidate.
//   k_collect        per row: candidates above that bin (random-k: key below ulo_l) are counted,
//                    the undecided ones are listed.
//   k_select         per segment: the exact threshold among the listed candidates, then the
//                    message offset of every row.  Layouts with a very large k_l instead count
//                    and scan the rows' winners in k_rowcount and k_rowscan.
//   k_emit           per row: the winners in index order to the message and e = +0 there (where
//                    the pass already stored +0 at every candidate, random-k and dense top-k
//                    segments, the losing candidates get their values back instead).
// A top-k segment with fewer than k_l candidates, or whose candidates do not fit the workspace, is
// collected again at a lower threshold (k_resolve sets it, k_collect re-reads the rows); only if
// that falls short too, or for random-k, is it resolved exactly over all of its elements by
// k_select.  Random-k's selection can also run without data, ahead of the step (the keys depend
// only on seed, step and position); the step is then one streaming pass (k_randk_apply).
// Block-random-k is one fused streaming pass (k_randblock_step).  The aggregates (Algorithm 1) sum
// each output element over the workers in worker order: in registers for block messages, in an
// LDS tile for sparse ones.
#pragma once

#include "ef_device.h"

namespace efs {

struct WSel {
  uint32_t* diag;      // [4]  diagnostics bits
  uint32_t* res;       // [L][kResWords] per-segment selection record
  uint32_t* hist;      // [L][kHCopies][kHBins] candidate histogram per segment, in copies that
                       // spread the atomics of concurrent rows
  uint32_t* samp;      // [nruns * kSampleRun] top-k sample keys
  uint32_t* counts;    // [nrows] candidates per row
  uint32_t* rcnt;      // [nrows] winners per row
  uint32_t* roff;      // [nrows] message position of each row's first winner
  uint32_t* rtie;      // [nrows] top-k: elements equal to the key A (counted, not stored)
  uint32_t* lcnt;      // [L][kSubLists][kLineWords] sizes of the sub-lists, one cache line each
  uint32_t* coff;      // [nrows] first entry of each row's candidates in the pool (kDropped: not
                       //   stored); one segment: written only for rows beyond their static slot
  uint32_t* pcnt;      // [kPools][kLineWords] fill counters of the overflow pool's parts
  uint32_t* cand_idx;  // [pool0 + capB] candidate pool: each row's static slot (soff, S),
  float* cand_val;     //   then the overflow pool for rows with more candidates (index order per row)
  uint32_t* cand_key;  //   key' of each candidate
  uint32_t* list_idx;  // sub-lists of undecided candidates, per segment (see SubLists)
  uint32_t* list_key;
  uint2* pairs;        // random-k, direct layouts: each row's undecided (key', index) pairs at its
                       //   pool entries (the list arrays' memory)
  const uint32_t* soff;  // [nrows+1] first entry of each row's static slot (several segments)
  uint32_t S;          // one segment: static slot entries per row (row r's slot starts at r * S and
                       //   holds min(S, the row's elements))
  uint32_t pool0;      // first entry of the overflow pool (the static slots end there)
  uint32_t capB;       // overflow pool entries, kPools equal parts (row r reserves in part r % kPools)
};

constexpr uint32_t kDropped = 0xFFFFFFFFu;  // coff of a row whose candidates did not fit
constexpr uint32_t kAccRow = 0x80000000u;   // counts flag of a top-k row emitted from acc (winning
                                            //   ties); the count is then the row's length
constexpr int kPools = 16;                  // parts of the overflow pool, one counter each

__device__ __forceinline__ uint32_t* res_of(const WSel& w, int l) { return w.res + (size_t)l * kResWords; }

// Several workers' steps in one launch of a selection kernel: worker blockIdx.y's buffers.  The
// gradient and residual of each worker are separate allocations (pointer tables); workspaces and
// messages lie at fixed strides from worker 0's.
constexpr int kBatchMax = 64;  // workers per launch of the selection kernels
struct Batch {
  uint64_t ws;                   // bytes between the workers' workspaces
  uint32_t msg;                  // entries between the workers' messages
  const void* g[kBatchMax];      // each worker's gradient (null: compress only)
  const float* src[kBatchMax];   // each worker's input: the residual e (fused steps) or acc
  float* e[kBatchMax];           // each worker's residual to update (null: compress only)
  uint32_t seed_lo[kBatchMax], seed_hi[kBatchMax];  // random-k: each worker's seed
};

template <typename P>
__device__ __forceinline__ P* shifted(P* p, uint64_t bytes) {
  return p ? reinterpret_cast<P*>(reinterpret_cast<uint8_t*>(const_cast<void*>(static_cast<const void*>(p))) + bytes)
           : p;
}

__device__ __forceinline__ WSel ws_at(WSel w, uint64_t off) {
  if (off == 0) return w;
  w.diag = shifted(w.diag, off);
  w.res = shifted(w.res, off);
  w.hist = shifted(w.hist, off);
  w.samp = shifted(w.samp, off);
  w.counts = shifted(w.counts, off);
  w.rcnt = shifted(w.rcnt, off);
  w.roff = shifted(w.roff, off);
  w.rtie = shifted(w.rtie, off);
  w.lcnt = shifted(w.lcnt, off);
  w.coff = shifted(w.coff, off);
  w.pcnt = shifted(w.pcnt, off);
  w.cand_idx = shifted(w.cand_idx, off);
  w.cand_val = shifted(w.cand_val, off);
  w.cand_key = shifted(w.cand_key, off);
  w.list_idx = shifted(w.list_idx, off);
  w.list_key = shifted(w.list_key, off);
  w.pairs = shifted(w.pairs, off);
  return w;  // (soff is a layout table: not shifted)
}

constexpr int kLineWords = 32;  // 128-byte L2 line: counters hit by many atomics get a line each
__device__ __forceinline__ uint32_t* lcnt_of(const WSel& w, int l, uint32_t c) {
  return w.lcnt + ((size_t)l * kSubLists + c) * kLineWords;
}
__device__ __forceinline__ uint32_t* pcnt_of(const WSel& w, uint32_t part) { return w.pcnt + (size_t)part * kLineWords; }

// Reserves n pool entries for row `row` (more than its static slot holds) in part row % kPools of
// the overflow pool; kDropped if the part is full.  One thread.
__device__ __forceinline__ uint32_t pool_reserve(const WSel& w, uint32_t row, uint32_t n) {
  const uint32_t part = row % kPools, q = w.capB / kPools;
  const uint32_t at = atomicAdd(pcnt_of(w, part), n);
  if (at > q || n > q - at) return kDropped;
  return w.pool0 + part * q + at;
}

// The first pool entry of a row holding cnt candidates, given its coff word co: one segment: its
// static slot unless they did not fit there.
__device__ __forceinline__ uint32_t row_entry(const Tables& T, const WSel& w, uint32_t row, uint32_t cnt,
                                              uint32_t co) {
  if (T.L > 1) return co;
  return cnt > min(w.S, (uint32_t)T.d - row * kTile) ? co : row * w.S;
}

// The static slot of a row: first entry and capacity.
__device__ __forceinline__ void static_slot(const Tables& T, const WSel& w, uint32_t row, uint32_t& at, uint32_t& cap) {
  if (T.L == 1) {  // every row but the last is a whole tile
    at = row * w.S;
    cap = min(w.S, (uint32_t)T.d - row * kTile);
  } else {
    at = w.soff[row];
    cap = w.soff[row + 1] - at;
  }
}

// First entry of sub-list c of segment l: sub-list c owns seg_lq[l] entries of the segment's region
// (loaded once per row, ahead of the row's loop).
__device__ __forceinline__ size_t sublist_base(const Tables& T, int l, uint32_t c) {
  return (size_t)T.seg_lbase[l] + (size_t)c * (uint32_t)T.seg_lq[l];
}

// The sub-lists of one segment read as one array of M[kSubLists] entries (any order).
struct SubLists {
  const uint32_t* arr;
  size_t base;  // the segment's list region
  uint32_t q;   // entries per sub-list
  uint32_t M[kSubLists + 1];  // M[c]: entries in sub-lists before c
  __device__ __forceinline__ uint32_t operator[](uint32_t f) const {
    uint32_t c = 0, b = 0;
#pragma unroll
    for (int x = 1; x < kSubLists; ++x) {
      if (f >= M[x]) {
        c = (uint32_t)x;
        b = M[x];
      }
    }
    return arr[base + (size_t)c * q + (f - b)];
  }
};

// ---------------------------------------------------------------------------------------------
// Utility kernels
// ---------------------------------------------------------------------------------------------
// The plain streaming kernels take one float4 group per thread in 64-thread workgroups (kRbTile
// elements each): short-lived workgroups keep the end of the grid short, where a streaming pass
// otherwise loses bandwidth.  Measured for the fused block-random-k step on ResNet-50 flat: 64
// threads 47.2 us per step, 128: 48.2, 256: 48.6; four float4 groups per thread: about 50.5.
constexpr int kRbNT = 64;
constexpr uint32_t kRbTile = 4u * kRbNT;

__device__ __forceinline__ int group_extent(uint32_t i0, uint32_t hi) {
  return i0 < hi ? (int)min(4u, hi - i0) : 0;
}

// Algorithm 1 accumulate step: acc = g + e.
template <int GDT>
__global__ __launch_bounds__(kRbNT) void k_accumulate(int32_t d, const void* g, const float* e, float* acc) {
  const uint32_t lo = blockIdx.x * kRbTile, hi = min((uint32_t)d, lo + kRbTile);
  const uint32_t i0 = lo + threadIdx.x * 4u;
  const int nv = group_extent(i0, hi);
  float gv[4], ev[4], a[4];
  if (hi - lo == kRbTile) {  // whole group (every workgroup but the last)
    load4gf<GDT>(g, i0, gv);
    load4f(e, i0, ev);
  } else {
    load4g<GDT>(g, i0, nv, gv);
    load4(e, i0, nv, ev);
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) a[q] = gv[q] + ev[q];
  store4(acc, i0, nv, a);
}

__global__ __launch_bounds__(kRbNT) void k_copy(int32_t d, const float* src, float* dst) {
  const uint32_t lo = blockIdx.x * kRbTile, hi = min((uint32_t)d, lo + kRbTile);
  const uint32_t i0 = lo + threadIdx.x * 4u;
  const int nv = group_extent(i0, hi);
  float v[4];
  if (hi - lo == kRbTile) load4f(src, i0, v);
  else load4(src, i0, nv, v);
  store4(dst, i0, nv, v);
}

// e[idx[j]] = +0 for every message entry (indices outside [0, d) are skipped).
__global__ __launch_bounds__(kNT) void k_sparse_zero(int32_t d, int32_t K, const uint32_t* idx, float* e) {
  const int j = blockIdx.x * kNT + threadIdx.x;
  if (j < K) {
    const uint32_t i = idx[j];
    if (i < (uint32_t)d) e[i] = 0.0f;
  }
}

// ---------------------------------------------------------------------------------------------
// Block-random-k (Section 3): one random start per segment, the run of k_l values after it.
// ---------------------------------------------------------------------------------------------
struct RunSeg {
  uint32_t o, n, k, P, s;
};

__device__ __forceinline__ RunSeg run_seg(const Tables& T, int l, uint32_t step, uint32_t s0, uint32_t s1) {
  RunSeg r;
  r.o = (uint32_t)T.seg_off[l];
  r.n = (uint32_t)T.seg_off[l + 1] - r.o;
  r.k = (uint32_t)T.seg_k[l];
  r.P = (uint32_t)T.seg_P[l];
  r.s = block_start((uint32_t)l, step, s0, s1, (uint32_t)T.seg_bl[l], (uint32_t)T.seg_nb[l]);
  return r;
}

// Position of element i within the run of its segment (>= k when not sent).
__device__ __forceinline__ uint32_t run_pos(const RunSeg& r, uint32_t i) {
  const uint32_t j = i - r.o;
  return j >= r.s ? j - r.s : j + r.n - r.s;
}

// The start of every segment that begins in [lo, hi) (segments sf..sl hold the data tile).  With
// one segment, its record rs is already loaded: no further load, which would make the
// workgroup's last wavefront wait for its stores before it ends (loads and stores share one
// counter).
__device__ __forceinline__ void write_starts(const Tables& T, int sf, int sl, const RunSeg& rs, uint32_t lo,
                                             uint32_t hi, uint32_t step, uint32_t s0, uint32_t s1,
                                             uint32_t* start) {
  if (sf == sl) {
    if (threadIdx.x == 0 && rs.o >= lo && rs.o < hi) start[sf] = rs.s;
    return;
  }
  for (int l = sf + (int)threadIdx.x; l <= sl; l += kRbNT) {
    const uint32_t ol = (uint32_t)T.seg_off[l];
    if (ol >= lo && ol < hi)
      start[l] = block_start((uint32_t)l, step, s0, s1, (uint32_t)T.seg_bl[l], (uint32_t)T.seg_nb[l]);
  }
}

// Fused worker step: acc = g + e; val[P_l + t] = acc on the run; e' = +0 on the run, acc elsewhere.
// One float4 group per thread for a float32 gradient (kRbTile elements per workgroup); two groups
// (kRbNT groups apart, each coalesced over the wavefront) for bf16, whose groups are 8-byte loads.
template <int GDT>
constexpr uint32_t rb_groups() { return GDT == 1 ? 2u : 1u; }
template <int GDT>
constexpr uint32_t rb_tile() { return kRbTile * rb_groups<GDT>(); }

template <int GDT>
__global__ __launch_bounds__(kRbNT) void k_randblock_step(Tables T, const void* g, float* e, uint32_t s0,
                                                        uint32_t s1, uint32_t step, uint32_t* start,
                                                        float* val) {
  if constexpr (GDT == 0) {
    const uint32_t lo = blockIdx.x * kRbTile, hi = min((uint32_t)T.d, lo + kRbTile);
    const uint32_t c = lo / kTile;  // the data tile holding this group: its first and last segment
    const int sf = T.chunk_sf[c], sl = T.chunk_sl[c];
    const uint32_t i0 = lo + threadIdx.x * 4u;
    const int nv = i0 < hi ? (int)min(4u, hi - i0) : 0;
    float gv[4], ev[4];
    if (hi - lo == kRbTile) {  // whole group (every workgroup but the last)
      load4gf<GDT>(g, i0, gv);
      load4f(e, i0, ev);
    } else {
      load4g<GDT>(g, i0, nv, gv);
      load4(e, i0, nv, ev);
    }
    RunSeg rs = run_seg(T, sf, step, s0, s1);
    int cur = sf;
    float out[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float a = gv[q] + ev[q];
      out[q] = a;
      if (q < nv) {
        const uint32_t i = i0 + q;
        if (sf != sl) {
          const int l = seg_of(i, sf, sl, T.seg_off);
          if (l != cur) {
            rs = run_seg(T, l, step, s0, s1);
            cur = l;
          }
        }
        const uint32_t t = run_pos(rs, i);
        if (t < rs.k) {
          val[rs.P + t] = a;
          out[q] = 0.0f;
        }
      }
    }
    store4(e, i0, nv, out);
    write_starts(T, sf, sl, rs, lo, hi, step, s0, s1, start);
  } else {
    constexpr uint32_t NG = rb_groups<GDT>(), TILE = rb_tile<GDT>();
    const uint32_t lo = blockIdx.x * TILE, hi = min((uint32_t)T.d, lo + TILE);
    const uint32_t c = lo / kTile;  // the data tile holding these groups: its first and last segment
    const int sf = T.chunk_sf[c], sl = T.chunk_sl[c];
    uint32_t i0[NG];
    int nv[NG];
#pragma unroll
    for (uint32_t r = 0; r < NG; ++r) {
      i0[r] = lo + (r * kRbNT + threadIdx.x) * 4u;
      nv[r] = i0[r] < hi ? (int)min(4u, hi - i0[r]) : 0;
    }
    float gv[NG][4], ev[NG][4];
    if (hi - lo == TILE) {  // whole tile (every workgroup but the last)
#pragma unroll
      for (uint32_t r = 0; r < NG; ++r) {
        load4gf<GDT>(g, i0[r], gv[r]);
        load4f(e, i0[r], ev[r]);
      }
    } else {
#pragma unroll
      for (uint32_t r = 0; r < NG; ++r) {
        load4g<GDT>(g, i0[r], nv[r], gv[r]);
        load4(e, i0[r], nv[r], ev[r]);
      }
    }
    RunSeg rs = run_seg(T, sf, step, s0, s1);
    int cur = sf;
#pragma unroll
    for (uint32_t r = 0; r < NG; ++r) {
      float out[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float a = gv[r][q] + ev[r][q];
        out[q] = a;
        if (q < nv[r]) {
          const uint32_t i = i0[r] + q;
          if (sf != sl) {
            const int l = seg_of(i, sf, sl, T.seg_off);
            if (l != cur) {
              rs = run_seg(T, l, step, s0, s1);
              cur = l;
            }
          }
          const uint32_t t = run_pos(rs, i);
          if (t < rs.k) {
            val[rs.P + t] = a;
            out[q] = 0.0f;
          }
        }
      }
      store4(e, i0[r], nv[r], out);
    }
    write_starts(T, sf, sl, rs, lo, hi, step, s0, s1, start);
  }
}

// Message position p -> segment (binary search over P).
__device__ __forceinline__ int seg_of_msg(uint32_t p, int L, const int32_t* P) { return seg_of(p, 0, L - 1, P); }

// compress_randblock: val[p] = acc at run position p; start[l] from the t = 0 entry.
__global__ __launch_bounds__(kNT) void k_randblock_gather(Tables T, int32_t K, const float* acc, uint32_t s0,
                                                          uint32_t s1, uint32_t step, uint32_t* start,
                                                          float* val) {
  const uint32_t p = blockIdx.x * kNT + threadIdx.x;
  if (p >= (uint32_t)K) return;
  const int l = seg_of_msg(p, T.L, T.seg_P);
  const RunSeg rs = run_seg(T, l, step, s0, s1);
  const uint32_t t = p - rs.P;
  uint32_t j = rs.s + t;
  if (j >= rs.n) j -= rs.n;
  val[p] = acc[rs.o + j];
  if (t == 0) start[l] = rs.s;
}

// In-place residual update for a block message: e[o_l + (s_l + t) mod d_l] = +0.
__global__ __launch_bounds__(kNT) void k_block_zero(Tables T, int32_t K, const uint32_t* start, float* e) {
  const uint32_t p = blockIdx.x * kNT + threadIdx.x;
  if (p >= (uint32_t)K) return;
  const int l = seg_of_msg(p, T.L, T.seg_P);
  const uint32_t o = T.seg_off[l], n = T.seg_off[l + 1] - o, t = p - T.seg_P[l];
  const uint32_t s = start[l] % n;
  uint32_t j = s + t;
  if (j >= n) j -= n;
  e[o + j] = 0.0f;
}

// Out-of-place residual update for a block message: e = +0 on the runs, acc elsewhere.  One float4
// group per thread (kRbTile elements per workgroup).
__global__ __launch_bounds__(kRbNT) void k_block_update(Tables T, const float* acc, const uint32_t* start, float* e) {
  const uint32_t lo = blockIdx.x * kRbTile, hi = min((uint32_t)T.d, lo + kRbTile);
  const uint32_t c = lo / kTile;  // the data tile holding this group: its first and last segment
  const int sf = T.chunk_sf[c], sl = T.chunk_sl[c];
  const uint32_t i0 = lo + threadIdx.x * 4u;
  const int nv = group_extent(i0, hi);
  float v[4];
  if (hi - lo == kRbTile) load4f(acc, i0, v);
  else load4(acc, i0, nv, v);
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if (q < nv) {
      const uint32_t i = i0 + q;
      const int l = sf == sl ? sf : seg_of(i, sf, sl, T.seg_off);
      const uint32_t o = T.seg_off[l], n = T.seg_off[l + 1] - o;
      const uint32_t s = start[l] % n, j = i - o;
      const uint32_t t = j >= s ? j - s : j + n - s;
      if (t < (uint32_t)T.seg_k[l]) v[q] = 0.0f;
    }
  }
  store4(e, i0, nv, v);
}

// ---------------------------------------------------------------------------------------------
// Aggregate (Algorithm 1): out = (sum over workers in order, from +0) / W, each output tile
// written once.
// ---------------------------------------------------------------------------------------------
// Output tiles of the sparse aggregate: kAggTile elements, summed by one wavefront (kAggRounds
// float4 groups per lane).
constexpr uint32_t kAggTile = 1024;  // 1024: 20.6 us on random-k messages; 2048: 23.8; 4096: 31.2
constexpr int kAggRounds = (int)kAggTile / (4 * 64);

// Column sum over W rows of K values (shared coordinates): sum_u v[u K + j] in row order from +0.0,
// loads of kSumBatch rows in flight together.
constexpr int kSumBatch = 8;
__device__ __forceinline__ float column_sum(const float* v, int32_t W, int32_t K, uint32_t j) {
  float s = 0.0f;
  for (int u0 = 0; u0 < W; u0 += kSumBatch) {
    float t[kSumBatch];
#pragma unroll
    for (int u = 0; u < kSumBatch; ++u) t[u] = u0 + u < W ? v[(size_t)(u0 + u) * K + j] : 0.0f;
#pragma unroll
    for (int u = 0; u < kSumBatch; ++u)
      if (u0 + u < W) s += t[u];
  }
  return s;
}

// tile_start[w * ts_stride + tau] = first entry of message w whose index lies in an aggregate tile
// >= tau (tau = 0..nt; an index >= d counts as tile nt).  Grid: (gx, W); each thread takes U
// entries at a time (coalesced, all loads in flight together) and the workgroups stride over the
// message: U = 1 with a thread per entry for short messages (the quickest form: one round), U = 8
// and a capped grid for long ones, so that 3.2e9 entries (32 messages of 1e8) do not need as many
// threads (1e9 elements at 1 %: 692 -> 450 us; at 10 %: 6.8 -> 3.8 ms).
// With `sums` (shared coordinates: W = 1 message whose values are vW workers' rows `vals`), entry
// j's thread also writes sums[j], the column sum of the rows in worker order.
// Entry j starts the tiles after its predecessor's tile, up to its own (past the last entry the
// tiles up to nt start at K).  A short run of tiles is written by its entry's thread; a longer one
// (a gap in a message crowded into a few layers) by the whole workgroup as one coalesced run, after
// each round (a thread writes its long run itself if the workgroup's list of them is full).
// For ascending messages the entries' runs partition 0..nt.
constexpr uint32_t kRunOwn = 32;        // runs of at most this many tiles are written by their own thread
                                        // (ResNet-50 top-k messages: 8.2 us with 128, 5.0 with 16-64)
constexpr int kRangeUBig = 8;           // entries per thread per round for long messages
constexpr int64_t kRangeBig = 1 << 22;  // total entries (W K) from which the long form is used
constexpr uint32_t kRangeStash = 512;   // long runs listed per workgroup and round

template <int kRangeU>
__global__ __launch_bounds__(kNT) void k_agg_ranges(int32_t d, int32_t K, int32_t nt, const uint32_t* idx,
                                                    uint32_t* tile_start, uint64_t ts_stride, const float* vals,
                                                    int32_t vW, float* sums) {
  __shared__ uint32_t s_nlong;
  __shared__ uint32_t s_ta[kRangeStash], s_n[kRangeStash], s_j[kRangeStash], s_own[kRangeStash];
  const int w = blockIdx.y;
  const uint32_t* m = idx + (size_t)w * K;
  uint32_t* ts = tile_start + (size_t)w * ts_stride;
  const size_t tbase = (size_t)w * ts_stride;
  auto tile = [&](uint32_t i) -> uint32_t { return i < (uint32_t)d ? i / kAggTile : (uint32_t)nt; };
  // tile tau of entry e's run starts at e, except past the last entry's own tile (at K)
  auto value = [&](uint32_t e, uint32_t tau, uint32_t e_own) -> uint32_t {
    return e == (uint32_t)K - 1u && tau > e_own ? (uint32_t)K : e;
  };
  if (threadIdx.x == 0) s_nlong = 0;
  __syncthreads();
  const uint32_t round = gridDim.x * (uint32_t)kNT * (uint32_t)kRangeU;
  for (uint32_t j0 = blockIdx.x * (uint32_t)kNT * (uint32_t)kRangeU; j0 < (uint32_t)K; j0 += round) {
    // each entry and its predecessor: the predecessor is the previous lane's entry (a shuffle);
    // only a wavefront's first lane loads it (a second load of every entry doubled the requests
    // this pass makes of the caches: 1e8 elements, 16 messages at 10 %: 192 -> 146 us)
    uint32_t cur[kRangeU], prv[kRangeU];
    const bool first = (threadIdx.x & 63u) == 0u;
#pragma unroll
    for (int u = 0; u < kRangeU; ++u) {
      const uint32_t j = j0 + (uint32_t)u * kNT + threadIdx.x;
      cur[u] = j < (uint32_t)K ? m[j] : 0u;
      prv[u] = first && j < (uint32_t)K && j > 0 ? m[j - 1] : 0u;
    }
#pragma unroll
    for (int u = 0; u < kRangeU; ++u) {
      const uint32_t up = __shfl_up(cur[u], 1u, 64);
      if (!first) prv[u] = up;
    }
    // shared coordinates (one message for vW workers): also the column sums of their values
    if (sums && w == 0) {
#pragma unroll
      for (int u = 0; u < kRangeU; ++u) {
        const uint32_t j = j0 + (uint32_t)u * kNT + threadIdx.x;
        if (j < (uint32_t)K) sums[j] = column_sum(vals, vW, K, j);
      }
    }
#pragma unroll
    for (int u = 0; u < kRangeU; ++u) {
      const uint32_t j = j0 + (uint32_t)u * kNT + threadIdx.x;
      if (j >= (uint32_t)K) continue;
      const uint32_t own = tile(cur[u]);
      const uint32_t ta = j == 0 ? 0u : tile(prv[u]) + 1u;
      const uint32_t tb = j == (uint32_t)K - 1u ? (uint32_t)nt : own;
      const uint32_t n = tb + 1u > ta ? tb + 1u - ta : 0u;
      bool mine = n <= kRunOwn;
      if (!mine) {
        const uint32_t p = atomicAdd(&s_nlong, 1u);
        if (p < kRangeStash) {
          s_ta[p] = ta;
          s_n[p] = n;
          s_j[p] = j;
          s_own[p] = own;
        } else {
          mine = true;
        }
      }
      if (mine)
        for (uint32_t k = 0; k < n; ++k) ts[ta + k] = value(j, ta + k, own);
    }
    __syncthreads();
    const uint32_t nl = min(s_nlong, kRangeStash);
    for (uint32_t q = 0; q < nl; ++q) {
      const uint32_t qa = s_ta[q], qe = qa + s_n[q], qj = s_j[q], qown = s_own[q];
      // 16-byte stores over the part of the run aligned in memory, single words at its two ends
      const uint32_t a4 = min(qe, qa + (uint32_t)((4u - (tbase + qa) % 4u) % 4u));
      const uint32_t b4 = a4 + (qe - a4) / 4u * 4u;
      if (threadIdx.x < a4 - qa) ts[qa + threadIdx.x] = value(qj, qa + threadIdx.x, qown);
      if (threadIdx.x < qe - b4) ts[b4 + threadIdx.x] = value(qj, b4 + threadIdx.x, qown);
      for (uint32_t o = a4 + 4u * threadIdx.x; o < b4; o += 4u * kNT) {
        const uint4 v = make_uint4(value(qj, o, qown), value(qj, o + 1, qown), value(qj, o + 2, qown),
                                   value(qj, o + 3, qown));
        *reinterpret_cast<uint4*>(ts + o) = v;
      }
    }
    __syncthreads();
    if (threadIdx.x == 0) s_nlong = 0;
    __syncthreads();
  }
}

// Workgroups of the range pass per message: one per kNT * U entries, capped for long messages so
// that all messages together fill the chip a few times over.
inline bool agg_ranges_big(int32_t K, int32_t W) { return (int64_t)K * W >= kRangeBig; }
inline uint32_t agg_ranges_gx(int32_t K, int32_t W) {
  if (!agg_ranges_big(K, W)) return (uint32_t)(((int64_t)K + kNT - 1) / kNT);
  const uint32_t need = (uint32_t)(((int64_t)K + kNT * kRangeUBig - 1) / (kNT * kRangeUBig));
  const uint32_t cap = (uint32_t)std::max<int32_t>(1, 8192 / std::max<int32_t>(W, 1));
  return std::max<uint32_t>(1u, std::min(need, cap));
}

// out = sum / W in IEEE float32.  For W a power of two the quotient is the exact scaling
// sum * (1 / W), which rounds identically (both are the one correctly rounded result of the same
// real number), and a multiply costs one instruction instead of a division sequence.
__device__ __forceinline__ float agg_scale(float sum, int32_t W, bool pow2, float inv) {
  return pow2 ? sum * inv : __fdiv_rn(sum, (float)W);
}

// Output stage of the aggregates.  q = the worker sum, divided by wdiv when averaging.  q goes to
// `out` when given; when `x` is given, Algorithm 1's parameter update is applied in the same pass:
// d = q (+ wd x when wd != 0); with a momentum buffer m: m = beta m + d, d = m; then x = x - d
// (each float32 operation rounded on its own).
struct AggOut {
  float* out;     // the aggregate, or nullptr
  float* x;       // parameters to update, or nullptr
  float* m;       // momentum buffer, or nullptr
  float beta, wd;
  int32_t wdiv;   // divisor of the average: the number of workers
  int32_t average;
};

__device__ __forceinline__ void agg_emit4(const AggOut& O, uint32_t i0, int nv, const float sum[4]) {
  const bool pow2 = (O.wdiv & (O.wdiv - 1)) == 0;
  const float inv = 1.0f / (float)O.wdiv;  // exact when wdiv is a power of two
  float q[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) q[j] = O.average ? agg_scale(sum[j], O.wdiv, pow2, inv) : sum[j];
  if (O.out) store4(O.out, i0, nv, q);
  if (O.x) {
    float x[4], m[4];
    load4(O.x, i0, nv, x);
    if (O.m) load4(O.m, i0, nv, m);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      float dj = q[j];
      if (O.wd != 0.0f) dj = dj + O.wd * x[j];
      if (O.m) {
        m[j] = O.beta * m[j] + dj;
        dj = m[j];
      }
      x[j] = x[j] - dj;
    }
    store4(O.x, i0, nv, x);
    if (O.m) store4(O.m, i0, nv, m);
  }
}

constexpr int kAggChunk = 4;        // sparse aggregate: entries per lane loaded together past the first 64
constexpr int kAggClaim = 256;      // sparse aggregate: claim slots (positions hash to x mod 256)

// Sparse aggregate: one wavefront per workgroup and one output tile of kAggTile elements per
// workgroup; many small workgroups resident per CU overlap each other's two load round trips
// (the tile's ranges, then its entries).  Lane j of a group of up to 64 workers holds worker
// j's entry range in the tile.  A tile no message enters is stored as zeros at once.  Otherwise
// its sums build up in an LDS tile: the tile's entries, in worker order, are added 64 at a time;
// lanes whose entries share a position add one after another in lane order (the lowest lane that
// still has to add claims the position's slot with an LDS atomic minimum; positions sharing a slot
// only wait for each other), which is worker order.  Entries past the first 64 are loaded
// kAggChunk per lane at a time.
struct AggLds {
  alignas(16) float acc[kAggTile];  // read and written as float4 groups
  uint32_t claim[kAggClaim];  // ~0 between adds
  uint32_t pre[65];           // entry prefix of each worker of the group
  uint32_t a[64];             // each worker's first entry in the tile
};

// Staged entry f of a worker group -> message entry: binary search of the prefixes.
__device__ __forceinline__ size_t agg_entry(const AggLds& S, int nw, int w0, int32_t K, uint32_t f) {
  int lo = 0, hi = nw - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (S.pre[mid] <= f) lo = mid; else hi = mid - 1;
  }
  return (size_t)(w0 + lo) * K + S.a[lo] + (f - S.pre[lo]);
}

// Prefixes of the worker group [w0, w0 + nw) whose ranges lane j holds (unclamped); returns the
// group's entry count.  Wave-uniform.
__device__ __forceinline__ uint32_t agg_group(AggLds& S, int nw, int32_t K, uint32_t ra, uint32_t rb) {
  const int lane = threadIdx.x;
  ra = min(ra, (uint32_t)K);
  rb = min(rb, (uint32_t)K);
  const uint32_t c = lane < nw && rb > ra ? rb - ra : 0u;
  const uint32_t inc = wave_incl_scan(c);
  S.pre[lane] = inc - c;
  S.a[lane] = ra;
  if (lane == 63) S.pre[64] = inc;
  __syncthreads();  // a one-wavefront workgroup: orders the LDS writes above before the reads
  return __shfl(inc, 63, 64);
}

// Adds one batch of up to 64 entries (lane order = worker order) into the LDS tile.
__device__ __forceinline__ void agg_add(AggLds& S, uint32_t lo, uint32_t hi, uint32_t i, float v, bool ok) {
  const uint32_t lane = threadIdx.x;
  bool pending = ok && i >= lo && i < hi;
  const uint32_t x = pending ? i - lo : 0u, c = x % kAggClaim;
  while (__ballot(pending)) {
    if (pending) atomicMin(&S.claim[c], lane);
    __syncthreads();
    if (pending && S.claim[c] == lane) {
      S.acc[x] += v;
      S.claim[c] = ~0u;
      pending = false;
    }
    __syncthreads();
  }
}

// Adds entries [f0, E) of the group set up by agg_group, kAggChunk per lane at a time.
__device__ __forceinline__ void agg_add_rest(AggLds& S, int nw, int w0, int32_t K, const uint32_t* idx,
                                             const float* val, uint32_t lo, uint32_t hi, uint32_t f0, uint32_t E) {
  for (; f0 < E; f0 += 64u * kAggChunk) {
    uint32_t ci[kAggChunk];
    float cv[kAggChunk];
#pragma unroll
    for (int u = 0; u < kAggChunk; ++u) {
      const uint32_t f = f0 + (uint32_t)u * 64u + threadIdx.x;
      const size_t j = f < E ? agg_entry(S, nw, w0, K, f) : 0;
      ci[u] = idx[j];
      cv[u] = val[j];
    }
#pragma unroll
    for (int u = 0; u < kAggChunk; ++u) agg_add(S, lo, hi, ci[u], cv[u], f0 + (uint32_t)u * 64u + threadIdx.x < E);
  }
}

// Tiles whose workers hold more than this many entries each on average add them worker by worker
// (agg_add_workers; 1e8 elements, 16 workers at 10 %: 414 -> 367 us, while at 1 %, about 10
// entries per worker and tile, the staged form is twice as fast).
constexpr uint32_t kAggDense = 48;
constexpr int kAggW = 16;  // dense tiles: chunks of 64 entries loaded together

// Dense tiles: the group's workers one after another, in order.  A message holds each position at
// most once, so the adds of one worker never collide: a chunk of up to 64 of one worker's entries
// is added by its lanes at once, with no claims and no barriers (the one wavefront's LDS accesses
// take effect in program order, so a position's adds run in worker order).  The chunks (worker by
// worker, 64 entries each) are numbered through a prefix over the workers' chunk counts; kAggW
// chunks are loaded together (coalesced), then added in order.
__device__ __forceinline__ void agg_add_workers(AggLds& S, int nw, int w0, int32_t K, const uint32_t* idx,
                                                const float* val, uint32_t lo, uint32_t hi) {
  const uint32_t lane = threadIdx.x;
  const uint32_t n = lane < (uint32_t)nw ? S.pre[lane + 1] - S.pre[lane] : 0u;  // worker `lane`'s entries
  const uint32_t a = S.a[lane];
  const uint32_t ch = (n + 63u) / 64u, chi = wave_incl_scan(ch);
  const uint32_t cpre = chi - ch;  // first chunk of worker `lane`
  const uint32_t nch = __shfl(chi, 63, 64);
  for (uint32_t q0 = 0; q0 < nch; q0 += kAggW) {
    uint32_t ci[kAggW];
    float cv[kAggW];
#pragma unroll
    for (int u = 0; u < kAggW; ++u) {
      const uint32_t q = q0 + (uint32_t)u;
      // chunk q's worker: the last one whose chunks start at or before q (wave-uniform)
      const int w = (int)__popcll(__ballot(lane < (uint32_t)nw && cpre <= q)) - 1;
      const uint32_t f = (q - __shfl(cpre, w, 64)) * 64u + lane;
      const bool ok = q < nch && f < __shfl(n, w, 64);
      const size_t j = (size_t)(w0 + w) * K + __shfl(a, w, 64) + f;
      ci[u] = ok ? idx[j] : 0u;
      cv[u] = ok ? val[j] : 0.0f;
      if (!ok) ci[u] = hi;  // adds nothing below
    }
#pragma unroll
    for (int u = 0; u < kAggW; ++u)
      if (ci[u] >= lo && ci[u] < hi) S.acc[ci[u] - lo] += cv[u];
  }
}

// Workgroup b -> tile: workgroups are dispatched to the 8 XCDs in turn (b mod 8), so XCD x is
// given chunks of kXcdChunk contiguous tiles in turn (chunks x, x + 8, ...), and the tiles past
// the last whole round of chunks in one contiguous part (a bijection for any n).  Neighbouring
// tiles share the cache lines of the range table and of the messages, and, within a chunk, an L2;
// the chunks spread a cluster of crowded tiles (top-k messages) over all the XCDs, where one
// contiguous eighth of the tiles per XCD left one XCD with most of the work.
constexpr uint32_t kXcds = 8;
constexpr uint32_t kXcdChunk = 32;
__device__ __forceinline__ uint32_t xcd_tile(uint32_t b, uint32_t n) {
  const uint32_t x = b % kXcds, j = b / kXcds;
  const uint32_t full = n / (kXcds * kXcdChunk) * kXcdChunk;  // each XCD's workgroups in whole rounds
  if (j < full) return ((j / kXcdChunk) * kXcds + x) * kXcdChunk + j % kXcdChunk;
  const uint32_t base = full * kXcds, rn = n - base, q = rn / kXcds, r = rn % kXcds;
  return base + x * q + min(x, r) + (j - full);
}

__global__ __launch_bounds__(64) void k_agg_sparse(int32_t d, int32_t W, int32_t K, int32_t nt,
                                                   const uint32_t* idx, const float* val,
                                                   const uint32_t* tile_start, AggOut O) {
  __shared__ AggLds S;
  const int lane = threadIdx.x;
  const uint32_t t = xcd_tile(blockIdx.x, (uint32_t)nt);  // the grid has exactly nt workgroups
  const uint32_t lo = t * kAggTile, hi = min((uint32_t)d, lo + kAggTile);
  // ranges of the first worker group (lane j: worker j; lanes past W read worker W - 1's)
  const int nw0 = min(W, 64);
  const uint32_t* ts = tile_start + (size_t)min(lane, nw0 - 1) * (nt + 1) + t;
  const uint32_t ra = ts[0], rb = ts[1];
  for (uint32_t x = lane; x < kAggClaim; x += 64) S.claim[x] = ~0u;
  const uint32_t E = agg_group(S, nw0, K, ra, rb);
  if (W <= 64 && E == 0) {
#pragma unroll
    for (int r = 0; r < kAggRounds; ++r) {
      const uint32_t i0 = lo + (uint32_t)(r * 64 + lane) * 4u;
      const int n = i0 < hi ? (int)min(4u, hi - i0) : 0;
      const float z[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      agg_emit4(O, i0, n, z);
    }
    return;
  }
#pragma unroll
  for (int r = 0; r < kAggRounds; ++r) {
    const f4 z = {0.0f, 0.0f, 0.0f, 0.0f};
    *reinterpret_cast<f4*>(&S.acc[(r * 64 + lane) * 4]) = z;
  }
  __syncthreads();
  if (E > kAggDense * (uint32_t)nw0) agg_add_workers(S, nw0, 0, K, idx, val, lo, hi);
  else agg_add_rest(S, nw0, 0, K, idx, val, lo, hi, 0u, E);
  for (int w0 = 64; w0 < W; w0 += 64) {  // further worker groups
    const int nw = min(64, W - w0);
    const uint32_t* tg = tile_start + (size_t)(w0 + min(lane, nw - 1)) * (nt + 1) + t;
    const uint32_t Eg = agg_group(S, nw, K, tg[0], tg[1]);
    if (Eg > kAggDense * (uint32_t)nw) agg_add_workers(S, nw, w0, K, idx, val, lo, hi);
    else agg_add_rest(S, nw, w0, K, idx, val, lo, hi, 0u, Eg);
  }
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kAggRounds; ++r) {
    const uint32_t x = (uint32_t)(r * 64 + lane) * 4u;
    const uint32_t i0 = lo + x;
    const int n = i0 < hi ? (int)min(4u, hi - i0) : 0;
    const f4 s4 = *reinterpret_cast<const f4*>(&S.acc[x]);
    const float v[4] = {s4.x, s4.y, s4.z, s4.w};
    agg_emit4(O, i0, n, v);
  }
}

// Single-segment layouts (flat scope): one workgroup per tile of R float4 groups per thread, no
// tables to look up and no barrier.  Each wavefront loads the starts of 64 workers at a time
// (lane j: worker wb + j), finds those whose run meets the tile with one ballot and visits them in
// ascending order.
template <int R>
__global__ __launch_bounds__(kNT) void k_agg_block1(int32_t d, int32_t W, int32_t K, const uint32_t* start,
                                                    const float* val, AggOut O) {
  constexpr uint32_t kT = (uint32_t)R * 4u * kNT;
  const uint32_t lo = blockIdx.x * kT, hi = min((uint32_t)d, lo + kT);
  const uint32_t n = (uint32_t)d, k = (uint32_t)K;
  const int lane = threadIdx.x & 63;
  float a[R][4];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int q = 0; q < 4; ++q) a[r][q] = 0.0f;
  for (int wb = 0; wb < W; wb += 64) {
    const int nw = min(64, W - wb);
    uint32_t s = 0;
    bool hit = false;
    if (lane < nw) {
      s = start[wb + lane] % n;
      const uint32_t e1 = min(s + k, n);
      // run piece 1: [s, e1); piece 2 (wrapped): [0, s + k - e1), empty unless the run wraps
      hit = max(lo, s) < min(hi, e1) || lo < min(hi, s + k - e1);
    }
    uint64_t todo = __ballot(hit);
    while (todo) {
      const int j = __ffsll((long long)todo) - 1;
      todo &= todo - 1;
      const uint32_t sw = __shfl(s, j, 64);
      const float* v = val + (size_t)(wb + j) * K;
      // piece 1 ends at e1 = min(s + k, n); piece 2 ([0, s + k - e1)) is empty unless the run wraps
      const uint32_t e1 = min(sw + k, n);
      const uint32_t a1 = max(lo, sw), b1 = min(hi, e1), b2 = min(hi, sw + k - e1);
#pragma unroll
      for (int r = 0; r < R; ++r) {
        const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const uint32_t i = i0 + q;
          if (i >= a1 && i < b1) a[r][q] += v[i - sw];
          else if (i < b2) a[r][q] += v[i + n - sw];
        }
      }
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r) {
    const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    const int nv = i0 < hi ? (int)min(4u, hi - i0) : 0;
    agg_emit4(O, i0, nv, a[r]);
  }
}

// Output stage for the elements q of the group at i0 whose bit q is set in `mask` (any subset: a
// group that straddles a segment boundary is written in parts by the two segments' workgroups).
__device__ __forceinline__ void agg_emit4m(const AggOut& O, uint32_t i0, uint32_t mask, const float sum[4]) {
  if (mask == 0xFu) {
    agg_emit4(O, i0, 4, sum);
    return;
  }
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    if (!((mask >> q) & 1u)) continue;
    const float s1[4] = {sum[q], 0.0f, 0.0f, 0.0f};
    agg_emit4(O, i0 + (uint32_t)q, 1, s1);
  }
}

// Multi-segment layouts: one workgroup per (1024-element data tile, segment) pair with an element
// in common, listed by a table built with the layout; otherwise as k_agg_block1 within the
// segment: the segment's block starts of 64 workers at a time, the workers whose run meets the
// tile found with one ballot and visited in ascending order.  Each element gets at most one value
// per worker, and the tile's elements outside the segment belong to the other pairs of the tile.
constexpr uint32_t kAggBT = 4u * kNT;  // one float4 group per thread

__global__ __launch_bounds__(kNT) void k_agg_block(Tables T, int32_t W, int32_t K, const uint32_t* start,
                                                   const float* val, AggOut O) {
  static_assert(kBtWords == 8, "two 16-byte loads per record");
  const uint4* rec = reinterpret_cast<const uint4*>(T.btile) + 2u * blockIdx.x;
  const uint4 r0 = rec[0], r1 = rec[1];  // one round trip: no chain through the segment tables
  const int l = (int)r0.y;
  const uint32_t o = r0.z, n = r0.w, k = r1.x, P = r1.y;
  const uint32_t tlo = r0.x * kAggBT;
  const uint32_t lo = max(tlo, o), hi = min(tlo + kAggBT, o + n);
  const uint32_t i0 = tlo + threadIdx.x * 4u;
  const int lane = threadIdx.x & 63;
  float a[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int wb = 0; wb < W; wb += 64) {
    const int nw = min(64, W - wb);
    uint32_t s = 0;
    bool hit = false;
    if (lane < nw) {
      s = start[(size_t)(wb + lane) * T.L + l] % n;
      // run piece 1: [o + s, o + e1), e1 = min(s + k, n); piece 2 (wrapped): [o, o + s + k - e1),
      // empty unless the run wraps (written without a conditional, as in k_agg_block1)
      const uint32_t e1 = min(s + k, n);
      hit = max(lo, o + s) < min(hi, o + e1) || lo < min(hi, o + (s + k - e1));
    }
    uint64_t todo = __ballot(hit);
    while (todo) {
      const int j = __ffsll((long long)todo) - 1;
      todo &= todo - 1;
      const uint32_t sw = __shfl(s, j, 64);
      const float* v = val + (size_t)(wb + j) * K + P;
      const uint32_t e1 = min(sw + k, n);
      const uint32_t a1 = max(lo, o + sw), b1 = min(hi, o + e1), b2 = min(hi, o + (sw + k - e1));
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t i = i0 + (uint32_t)q;
        if (i >= a1 && i < b1) a[q] += v[i - o - sw];
        else if (i >= lo && i < b2) a[q] += v[i - o + n - sw];
      }
    }
  }
  uint32_t mask = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if (i0 + (uint32_t)q >= lo && i0 + (uint32_t)q < hi) mask |= 1u << q;
  if (mask) agg_emit4m(O, i0, mask, a);
}

// ---------------------------------------------------------------------------------------------
// Random-k with the selection prepared ahead: the keys depend only on the seed, the step and the
// position (Section 3, random-k), so the message indices can be chosen before the gradient
// exists.  The step is then one streaming pass, one workgroup per kAggTile-element tile (one
// float4 group per thread): acc = g + e; the tile's winners (entries [ts[t], ts[t + 1]) of the
// prepared message, in ascending order) take their values from acc, and e = acc with +0 there.
// ---------------------------------------------------------------------------------------------
static_assert(kAggTile == 4u * kNT, "one float4 group per thread");

template <int GDT>
__global__ __launch_bounds__(kNT) void k_randk_apply(int32_t d, int32_t K, const uint32_t* ts, const uint32_t* idx,
                                                     const void* g, float* e, float* val) {
  __shared__ __align__(16) int32_t slot[kAggTile];  // element -> its winner's message entry, or -1
  const uint32_t t = blockIdx.x, lo = t * kAggTile, hi = min((uint32_t)d, lo + kAggTile);
  const uint32_t i0 = lo + threadIdx.x * 4u;
  const uint32_t ja = ts[t], jb = min(ts[t + 1], (uint32_t)K);
  const bool whole = hi - lo == kAggTile;
  const int nv = i0 < hi ? (int)min(4u, hi - i0) : 0;
  float gv[4], ev[4];
  if (whole) {
    load4gf<GDT>(g, i0, gv);
    load4f(e, i0, ev);
  } else {
    load4g<GDT>(g, i0, nv, gv);
    load4(e, i0, nv, ev);
  }
  *reinterpret_cast<int4*>(&slot[threadIdx.x * 4u]) = make_int4(-1, -1, -1, -1);
  __syncthreads();
  for (uint32_t j = ja + threadIdx.x; j < jb; j += kNT) {
    const uint32_t x = idx[j] - lo;
    if (x < kAggTile) slot[x] = (int32_t)j;
  }
  __syncthreads();
  const int4 sl = *reinterpret_cast<const int4*>(&slot[threadIdx.x * 4u]);
  const int32_t s4[4] = {sl.x, sl.y, sl.z, sl.w};
  float a[4];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    a[q] = gv[q] + ev[q];
    if (s4[q] >= 0) {
      val[s4[q]] = a[q];
      a[q] = 0.0f;
    }
  }
  if (whole) store4(e, i0, 4, a);
  else store4(e, i0, nv, a);
}

// Shared block starts: the column sums of the W workers' values (worker order, from +0.0).
__global__ __launch_bounds__(kNT) void k_shared_sum(int32_t W, int32_t K, const float* val, float* sum) {
  const uint32_t j = blockIdx.x * kNT + threadIdx.x;
  if (j < (uint32_t)K) sum[j] = column_sum(val, W, K, j);
}

// Standard SGD's exchange (no compression): out = (sum over workers in order, from +0.0) / W of
// the dense gradients g[W][d].  Two float4 groups per thread, one in each half of the groups, and
// the loads of kDenseBatch workers in flight together (16 workers on ResNet-50's d: 287 us, 76 %
// of 8 TB/s, against 305 us with one group and 8 loads in flight, 296 us with one group and 16).
constexpr int kDenseBatch = 16;
__global__ __launch_bounds__(kNT) void k_dense_average(int32_t d, int32_t W, const float* g, int average,
                                                       float* out) {
  const uint32_t ngr = ((uint32_t)d + 3u) / 4u;
  const uint32_t half = (ngr + 1u) / 2u;
  const uint32_t t = blockIdx.x * kNT + threadIdx.x;
  if (t >= half) return;
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint32_t gi = t + (uint32_t)h * half;
    if (gi >= ngr) break;
    const uint32_t i0 = gi * 4u;
    const int nv = (int)min(4u, (uint32_t)d - i0);
    float s[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int w0 = 0; w0 < W; w0 += kDenseBatch) {
      float v[kDenseBatch][4];
#pragma unroll
      for (int u = 0; u < kDenseBatch; ++u)
        if (w0 + u < W) load4(g + (size_t)(w0 + u) * d, i0, nv, v[u]);
#pragma unroll
      for (int u = 0; u < kDenseBatch; ++u)
        if (w0 + u < W)
#pragma unroll
          for (int q = 0; q < 4; ++q) s[q] += v[u][q];
    }
    const bool pow2 = (W & (W - 1)) == 0;
    const float inv = 1.0f / (float)W;
    float o[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) o[q] = average ? agg_scale(s[q], W, pow2, inv) : s[q];
    store4(out, i0, nv, o);
  }
}

// ---------------------------------------------------------------------------------------------
// Selection pipeline (top-k, random-k)
// KIND 0 = top-k: key' = magnitude bits of the value, the k largest are sent.
// KIND 1 = random-k: key' = ~Philox key, so the k smallest random keys have the largest key'.
// Among equal key', lower indices are sent first.
// ---------------------------------------------------------------------------------------------
template <int KIND>
__device__ __forceinline__ uint32_t sel_key(uint32_t idx, float val, uint32_t o, int l, uint32_t step,
                                            uint32_t s0, uint32_t s1) {
  if constexpr (KIND == 0) return mag_key(val);
  else return ~randk_key(idx - o, (uint32_t)l, step, s0, s1);
}

constexpr int kBatch = 8;             // independent loads in flight per thread in the selection passes
constexpr uint32_t kListLds = 8192;    // listed candidates held in LDS by k_select
constexpr uint32_t kRowsLds = 16384;   // rows per segment whose list additions k_select counts in LDS
constexpr uint32_t kRankList = 256;    // lists up to this size are ranked directly (no radix levels)
constexpr uint32_t kBigK = 1u << 20;   // layouts with a k_l this large count row winners in parallel
constexpr int32_t kBigRows = 16384;    // ... and so do layouts with a segment of more rows than this
constexpr uint32_t kSelPer = 8;        // rows per k_select thread held in registers
constexpr uint32_t kHistDirect = 32;   // rows with more candidates histogram them in LDS first
constexpr int kHCopies = 16;           // copies of each candidate histogram (row r adds to copy r % 16)
constexpr uint32_t kDiagCount = 4u;    // diagnostics: the row counts of a segment did not add up to k_l
// R_IT of a top-k segment on a many-row layout whose threshold key T is shared by more listed
// candidates than win: k_rowcount counts each row's keys equal to T, k_rowscan finds the last
// winner among them (R_NEED of them win, in index order) and writes the real R_IT.
constexpr uint32_t kTieRows = 0xFFFFFFFEu;

// Workgroup-wide AND and OR of per-thread values; `lds` holds 2 * kSelNT / 64 words.
__device__ __forceinline__ void block_and_or(uint32_t& a, uint32_t& o, uint32_t* lds) {
#pragma unroll
  for (int s = 32; s > 0; s >>= 1) {
    a &= __shfl_xor(a, s, 64);
    o |= __shfl_xor(o, s, 64);
  }
  constexpr int nw = kSelNT / 64;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  if (lane == 0) {
    lds[wid] = a;
    lds[nw + wid] = o;
  }
  __syncthreads();
  a = 0xFFFFFFFFu;
  o = 0u;
#pragma unroll
  for (int w = 0; w < nw; ++w) {
    a &= lds[w];
    o |= lds[nw + w];
  }
  __syncthreads();
}

// Calls fn(f, keys[f]) for every f < n, in a strided order with kBatch loads in flight.
template <int B = kBatch, typename K, typename F>
__device__ __forceinline__ void for_keys(const K& keys, uint32_t n, F fn) {
  for (uint32_t base = 0; base < n; base += (uint32_t)kSelNT * B) {
    uint32_t k[B];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const uint32_t f = base + (uint32_t)u * kSelNT + threadIdx.x;
      k[u] = f < n ? keys[f] : 0u;
    }
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const uint32_t f = base + (uint32_t)u * kSelNT + threadIdx.x;
      if (f < n) fn(f, k[u]);
    }
  }
}

// A list in global memory, swept sub-list by sub-list: the position within a sub-list is the
// address, where indexing the concatenation searched the sub-list bounds for every key (BERT flat
// at 10 % with bf16 values: the selection kernel's sweeps of a 211,000-key list took 97 us that
// way, the whole kernel 77 us this way).  fn(f, key) gets the position f in the concatenation.
template <int B = kBatch, typename F>
__device__ __forceinline__ void for_keys(const SubLists& L, uint32_t n, F fn) {
  (void)n;  // = L.M[kSubLists]
  for (int c = 0; c < kSubLists; ++c) {
    uint32_t m0 = 0, m1 = 0;  // the bounds of sub-list c, selected without indexing M
#pragma unroll
    for (int x = 0; x <= kSubLists; ++x) {
      if (x == c) m0 = L.M[x];
      if (x == c + 1) m1 = L.M[x];
    }
    const uint32_t nc = m1 - m0;
    const uint32_t* a = L.arr + L.base + (size_t)c * L.q;
    for (uint32_t base = 0; base < nc; base += (uint32_t)kSelNT * B) {
      uint32_t k[B];
#pragma unroll
      for (int u = 0; u < B; ++u) {
        const uint32_t j = base + (uint32_t)u * kSelNT + threadIdx.x;
        k[u] = j < nc ? a[j] : 0u;
      }
#pragma unroll
      for (int u = 0; u < B; ++u) {
        const uint32_t j = base + (uint32_t)u * kSelNT + threadIdx.x;
        if (j < nc) fn(m0 + j, k[u]);
      }
    }
  }
}

// Exact selection over the whole segment (used when the candidates cannot contain the answer):
// radix levels over the keys of all d_l elements, then an index-ordered emission.
template <int KIND>
__device__ void slow_select(const Tables& T, int l, const float* data, float* e_zero, uint32_t* out_idx,
                            float* out_val, uint32_t s0, uint32_t s1, uint32_t step, uint32_t* hist, uint32_t* lds) {
  const uint32_t o = (uint32_t)T.seg_off[l], n = (uint32_t)T.seg_off[l + 1] - o;
  const uint32_t P = (uint32_t)T.seg_P[l], kl = (uint32_t)T.seg_k[l];
  // random-k keys depend on the position only: without data (a selection prepared ahead of the
  // step) only the indices are written
  auto keyat = [&](uint32_t j) -> uint32_t {
    return sel_key<KIND>(o + j, KIND == 1 && !data ? 0.0f : data[o + j], o, l, step, s0, s1);
  };
  uint32_t prefix = 0, need = kl;
  int known = 0;
  while (known < 32) {
    const int w = min(11, 32 - known);
    const int shift = 32 - known - w;
    for (int b = threadIdx.x; b < (1 << w); b += kSelNT) hist[b] = 0;
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < n; j += kSelNT) {
      const uint32_t k = keyat(j);
      if (known == 0 || (k >> (32 - known)) == (prefix >> (32 - known)))
        atomicAdd(&hist[(k >> shift) & ((1u << w) - 1u)], 1u);
    }
    __syncthreads();
    uint32_t above;
    const int bin = block_resolve<kSelNT>(hist, 1 << w, need, lds, above);
    prefix |= (uint32_t)max(bin, 0) << shift;
    need -= above;
    known += w;
  }
  const uint32_t Tk = prefix, r = need;
  uint32_t run_a = 0, run_b = 0;
  for (uint32_t j0 = 0; j0 < n; j0 += kSelNT) {
    const uint32_t j = j0 + threadIdx.x;
    uint32_t a = 0, b = 0;
    if (j < n) {
      const uint32_t k = keyat(j);
      a = k > Tk;
      b = k == Tk;
    }
    uint32_t tot;
    const uint32_t ex = block_excl_scan<kSelNT>(a | (b << 16), lds, tot);
    const uint32_t ea = run_a + (ex & 0xFFFFu), eb = run_b + (ex >> 16);
    if ((a || (b && eb < r)) && ea + min(eb, r) < kl) {
      const uint32_t pos = P + ea + min(eb, r);
      out_idx[pos] = o + j;
      if (out_val) out_val[pos] = data[o + j];
      if (e_zero) e_zero[o + j] = 0.0f;
    }
    run_a += tot & 0xFFFFu;
    run_b += tot >> 16;
  }
}

// ---------------------------------------------------------------------------------------------
// Workgroup helpers of the per-segment kernels (kSelNT threads)
// ---------------------------------------------------------------------------------------------
__device__ __forceinline__ uint32_t block_max_u32(uint32_t v, uint32_t* lds) {
#pragma unroll
  for (int s = 32; s > 0; s >>= 1) v = max(v, (uint32_t)__shfl_xor(v, s, 64));
  constexpr int nw = kSelNT / 64;
  if ((threadIdx.x & 63) == 0) lds[threadIdx.x >> 6] = v;
  __syncthreads();
  v = 0;
#pragma unroll
  for (int w = 0; w < nw; ++w) v = max(v, lds[w]);
  __syncthreads();
  return v;
}

// Position of the r-th (1-based) entry equal to x among keys[0, m), in position order.  Each
// wave owns a contiguous share of the positions; `lds` holds kSelNT / 64 words.
template <typename K>
__device__ __forceinline__ uint32_t block_nth_equal(const K& keys, uint32_t m, uint32_t x, uint32_t r, uint32_t* lds) {
  __shared__ uint32_t s_pos;
  constexpr int NW = kSelNT / 64;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const uint32_t W0 = (uint32_t)(((uint64_t)m * wid) / NW), W1 = (uint32_t)(((uint64_t)m * (wid + 1)) / NW);
  uint32_t cnt = 0;
  for (uint32_t b = W0; b < W1; b += 64) {
    const uint32_t f = b + lane;
    cnt += (uint32_t)__popcll(__ballot(f < W1 && keys[f] == x));
  }
  if (lane == 0) lds[wid] = cnt;
  if (threadIdx.x == 0) s_pos = m;
  __syncthreads();
  uint32_t before = 0;
  for (int w = 0; w < wid; ++w) before += lds[w];
  if (before < r && r <= before + cnt) {  // wave-uniform: this wave holds the r-th match
    uint32_t run = before;
    for (uint32_t b = W0; b < W1; b += 64) {
      const uint32_t f = b + lane;
      const bool t = f < W1 && keys[f] == x;
      const uint64_t mk = __ballot(t);
      const uint32_t c = (uint32_t)__popcll(mk);
      if (run + c >= r) {
        if (t && run + lanes_below(mk) + 1 == r) s_pos = f;
        break;
      }
      run += c;
    }
  }
  __syncthreads();
  const uint32_t p = s_pos;
  __syncthreads();
  return p;
}

// The r-th smallest idx[j] (r >= 1, indices distinct) among the j < m with keys[j] == x: radix
// levels over ~idx, whose largest values are the smallest indices.
template <typename K, typename I>
__device__ __forceinline__ uint32_t block_nth_smallest_tie(const K& keys, const I& idx, uint32_t m, uint32_t x,
                                           uint32_t r, uint32_t* hist, uint32_t* lds) {
  uint32_t prefix = 0, need = r;
  int known = 0;
  while (known < 32) {
    const int w = min(11, 32 - known);
    const int shift = 32 - known - w;
    for (int b = threadIdx.x; b < (1 << w); b += kSelNT) hist[b] = 0;
    __syncthreads();
    const uint32_t pmask = known == 0 ? 0u : (0xFFFFFFFFu << (32 - known));
    for (uint32_t j = threadIdx.x; j < m; j += kSelNT) {
      if (keys[j] == x) {
        const uint32_t v = ~idx[j];
        if ((v & pmask) == (prefix & pmask)) atomicAdd(&hist[(v >> shift) & ((1u << w) - 1u)], 1u);
      }
    }
    __syncthreads();
    uint32_t above;
    const int bin = block_resolve<kSelNT>(hist, 1 << w, need, lds, above);
    prefix |= (uint32_t)max(bin, 0) << shift;
    need -= above;
    known += w;
  }
  return ~prefix;
}

// Candidate histogram bin of a top-k key >= A (higher bins hold larger keys).  Bin 0 holds the
// key A alone, so that a threshold landing on a value shared by very many elements (exact zeros,
// say) is recognised as a pure tie; larger keys go to 1 + ((key - A - 1) >> sh), clamped to the
// last bin.
__device__ __forceinline__ uint32_t cand_bin(uint32_t key, uint32_t A, uint32_t sh) {
  return key == A ? 0u : 1u + min((key - A - 1u) >> sh, (uint32_t)kHBins - 2u);
}

// Magnitude keys of acc read in place (a row's elements equal to A are counted, not stored).
struct AccKeys {
  const float* p;
  __device__ __forceinline__ uint32_t operator[](uint32_t f) const { return mag_key(p[f]); }
};

// The first and one past the last element of a row.
__device__ __forceinline__ void row_bounds(const Tables& T, uint32_t row, uint32_t& lo, uint32_t& hi) {
  uint32_t o = 0, e_ = (uint32_t)T.d, tb = row * kTile;
  if (T.L > 1) {
    const uint4 rr = reinterpret_cast<const uint4*>(T.row_rec)[row];
    o = rr.y;
    e_ = rr.z;
    tb = rr.w;
  }
  lo = max(o, tb);
  hi = min(e_, tb + kTile);
}

// LDS histogram add of one key per active lane: the lanes whose bin is the first active lane's
// add together with one atomic, the others one by one.  Sample keys crowd a few bins (BERT's
// gradients: a histogram of 65,536 of them took 20 us with an atomic per key, same-address
// atomics of one wavefront being serialised; the sample selection 36 -> 28 us this way).
__device__ __forceinline__ void hist_add_peel(uint32_t* h, uint32_t b) {
  const uint32_t b0 = __builtin_amdgcn_readfirstlane(b);
  const uint64_t same = __ballot(b == b0);
  if (b != b0) atomicAdd(&h[b], 1u);
  else if ((threadIdx.x & 63u) == (uint32_t)(__ffsll((long long)same) - 1)) atomicAdd(&h[b0], (uint32_t)__popcll(same));
}

// ---------------------------------------------------------------------------------------------
// Top-k sample
// ---------------------------------------------------------------------------------------------
// One workgroup of kSampleRun threads per run: a segment of up to kExactMax elements is sampled
// whole (runs of consecutive positions).  A larger one, given s = runs * kSampleRun samples by the
// layout (a share of its samples in proportion to its size, at least kSampleMinRuns runs), is
// split into s strata of equal length (to within one element) and sampled once in each, at a
// pseudo-random position inside the stratum (stratified sampling): every part of the segment, a
// small tensor of large values inside a flat gradient included, is represented in proportion to
// its size, and the count of sampled keys above a value varies no more than a simple random
// sample's would (runs of contiguous elements, by contrast, sample a handful of clusters: a small
// tensor is either missed or over-represented many times).  Sample q = run * kSampleRun + thread;
// the runs of a sampled segment also clear its candidate histogram (kHCopies * kHBins words).
static_assert(kHCopies * kHBins == kSampleMax, "a sampled segment's histogram is cleared by its samples");
static_assert(kExactMax <= kSampleMax, "a segment sampled whole fits the sample keys held in LDS");
constexpr int kSampleKeysPer = kSampleMax / kSelNT;  // sample keys per thread, loaded in one round trip
static_assert(2 * kRankList <= kHBins, "the ranked entries (64-bit words) of an exact segment fit a histogram array");

// Positions 0, 1, ... as the indices of keys held in position order.
struct LocalPos {
  __device__ uint32_t operator[](uint32_t f) const { return f; }
};
template <typename K, typename I>
__device__ __forceinline__ void list_threshold_ao(const K& key, const I& idx, uint32_t m, uint32_t need,
                                                  uint32_t kand, uint32_t kor, uint32_t* hist, uint32_t* lds,
                                                  uint64_t* g, uint32_t& T_out, uint32_t& IT_out,
                                                  uint32_t* defer_need = nullptr);
template <int GDT, bool FUSED>
__global__ __launch_bounds__(kSampleRun) void k_sample_gather(Tables T, WSel ws0, Batch BT) {
  const WSel ws = ws_at(ws0, (uint64_t)blockIdx.y * BT.ws);
  const void* g = BT.g[blockIdx.y];
  const float* src = BT.src[blockIdx.y];
  const uint32_t r = blockIdx.x;
  // a table lookup: one round trip instead of a binary search's chain (none for one segment)
  const int l = T.L == 1 ? 0 : T.run_seg[r];
  const uint32_t o = (uint32_t)T.seg_off[l], n = (uint32_t)T.seg_off[l + 1] - o;
  const uint32_t q = r - (uint32_t)T.seg_ro[l];
  uint32_t i;
  bool in = true;
  if (n <= (uint32_t)kExactMax) {
    const uint32_t j = q * kSampleRun + threadIdx.x;
    in = j < n;
    i = o + j;
  } else {
    const uint32_t ns = ((uint32_t)T.seg_ro[l + 1] - (uint32_t)T.seg_ro[l]) * kSampleRun;  // samples
    const uint32_t sq = q * kSampleRun + threadIdx.x;  // the stratum
    const uint32_t a = (uint32_t)(((uint64_t)sq * n) / ns);
    const uint32_t b = (uint32_t)(((uint64_t)(sq + 1u) * n) / ns);
    const uint32_t x = philox(make_uint4(sq, 0u, 0u, kSampleTag | (uint32_t)l), 0u, 0u).x;
    i = o + a + __umulhi(x, b - a);  // uniform in [a, b): b > a because ns <= n (runs <= n / kSampleRun)
    for (uint32_t h = sq; h < (uint32_t)(kHCopies * kHBins); h += ns) ws.hist[(size_t)l * kHCopies * kHBins + h] = 0u;
  }
  // the overflow pool's counters start from zero (the first kernel of a top-k step)
  if (r == 0 && threadIdx.x < (unsigned)kPools) *pcnt_of(ws, threadIdx.x) = 0u;
  uint32_t key = 0;
  if (in) {
    float a;
    if constexpr (FUSED) a = load1g<GDT>(g, i) + src[i];
    else a = src[i];
    key = mag_key(a);
  }
  ws.samp[(size_t)r * kSampleRun + threadIdx.x] = key;
}

// Per segment (one workgroup) the candidate rule of the streaming pass:
//  * at most kExactMax elements: the exact k_l-th largest key T over the whole segment and the
//    bound I (one past the index of the last tie sent; ties go to lower indices); the candidates
//    are then exactly the winners (mode 1).
//  * larger segments: A = the lower edge of the bin of the top 11 key bits that holds the
//    srank-th largest sampled key (srank: the expected rank of the k_l-th key in the sample plus
//    a margin); every key >= A is a candidate.  The candidates are histogrammed in bins of 2^sh
//    keys above A, sh chosen so that the range up to the urank-th sampled key (the expected rank
//    minus the margin) spans about 1024 bins: the k_l-th key very likely falls inside it, and the
//    bins there are as narrow as the sample allows (mode 0).
__global__ __launch_bounds__(kSelNT) void k_sample_select(Tables T, WSel ws0, Batch BT) {
  const WSel ws = ws_at(ws0, (uint64_t)blockIdx.y * BT.ws);
  __shared__ uint32_t keys[kSampleMax];
  __shared__ uint32_t hist[kHBins];
  __shared__ __align__(8) uint32_t hist2[kHBins];
  __shared__ uint32_t lds[2 * kSelNT / 64];
  const int l = blockIdx.x;
  const uint32_t o = (uint32_t)T.seg_off[l], n = (uint32_t)T.seg_off[l + 1] - o;
  const uint32_t* sk = ws.samp + (size_t)T.seg_ro[l] * kSampleRun;
  uint32_t* R = res_of(ws, l);
  if (n <= (uint32_t)kExactMax) {
    uint32_t kand = 0xFFFFFFFFu, kor = 0u;
    for_keys<kSampleKeysPer>(sk, n, [&](uint32_t f, uint32_t k) {
      keys[f] = k;
      kand &= k;
      kor |= k;
    });
    block_and_or(kand, kor, lds);  // its barriers also publish keys[]
    // the k_l best of the segment's keys (positions as indices): hist2 holds the ranked entries
    uint32_t Tk, IT;
    list_threshold_ao(keys, LocalPos{}, n, (uint32_t)T.seg_k[l], kand, kor, hist, lds,
                      reinterpret_cast<uint64_t*>(hist2), Tk, IT);
    const uint32_t it = IT == 0xFFFFFFFFu ? IT : o + IT;  // every tie wins, or one past the last
    if (threadIdx.x == 0) {
      R[R_A] = Tk;
      R[R_IA] = it;
      R[R_T] = Tk;
      R[R_IT] = it;
      R[R_MODE] = 1;
      R[R_SLOW] = 0;
      R[R_OVF] = 0;
    }
    return;
  }
  // sampled: bins of the top 11 key bits (8 exponent + 3 mantissa bits); keys stay in registers
  const uint32_t ns = ((uint32_t)T.seg_ro[l + 1] - (uint32_t)T.seg_ro[l]) * kSampleRun;  // samples
  for (int b = threadIdx.x; b < kHBins; b += kSelNT) hist[b] = 0;
  __syncthreads();
  uint32_t kmax = 0u;
  // (the enlarged samples of dense layouts: the peeled add; a 16,384-key sample of ResNet-50's
  // gradients took 1 us longer with it than with an atomic per key)
  const bool peel = ns > (uint32_t)kSampleTotal;
  for_keys<kSampleKeysPer>(sk, ns, [&](uint32_t, uint32_t k) {
    if (peel) hist_add_peel(hist, k >> 20);
    else atomicAdd(&hist[k >> 20], 1u);
    kmax = max(kmax, k);
  });
  __syncthreads();
  kmax = block_max_u32(kmax, lds);
  // Key edge of the rank-th largest sampled key: the lower (or upper) edge of its top-11-bit bin,
  // refined by the next 11 bits when that bin holds more than 64 sampled keys (concentrated
  // values: an unrefined edge could take up to the whole bin's keys as candidates beyond the
  // rank, which the candidate pool is not sized for).  Both ranks' bins come from one scan of
  // the histogram.
  const uint32_t rank = (uint32_t)T.seg_srank[l], urank = (uint32_t)T.seg_urank[l];
  int bin_t, bin_u;
  uint32_t above_t, above_u;
  block_resolve2<kSelNT>(hist, kHBins, rank < ns ? rank : 0u, urank, lds, bin_t, above_t, bin_u, above_u);
  auto rank_edge = [&](int bin, uint32_t above, uint32_t rk, bool upper) -> uint32_t {
    if (bin < 0) return 0u;
    if (hist[bin] <= 64u) return ((uint32_t)bin + (upper ? 1u : 0u)) << 20;
    for (int b = threadIdx.x; b < kHBins; b += kSelNT) hist2[b] = 0;
    __syncthreads();
    for_keys(sk, ns, [&](uint32_t, uint32_t k) {
      if ((k >> 20) == (uint32_t)bin) atomicAdd(&hist2[(k >> 9) & (kHBins - 1)], 1u);
    });
    __syncthreads();
    uint32_t above2;
    const int bin2 = block_resolve<kSelNT>(hist2, kHBins, rk - above, lds, above2);
    return ((uint32_t)bin << 20) + (((uint32_t)max(bin2, 0) + (upper ? 1u : 0u)) << 9);
  };
  // rank >= sample size: every element is a candidate
  const uint32_t thr = rank < ns ? rank_edge(bin_t, above_t, rank, false) : 0u;
  // the bins resolve the range up to the upper edge of where the k-th key very likely lies
  uint32_t top = rank_edge(bin_u, above_u, urank, true);
  if (top <= thr || top > kmax) top = kmax;
  const uint32_t span = top - thr;
  const uint32_t sh = span < 1024u ? 0u : (uint32_t)(32 - __clz(span)) - 10u;
  if (threadIdx.x == 0) {
    R[R_A] = thr;
    R[R_IA] = 0xFFFFFFFFu;
    R[R_SH] = sh;
    R[R_MODE] = 0;
    R[R_SLOW] = 0;
    R[R_OVF] = 0;
  }
}

// ---------------------------------------------------------------------------------------------
// Streaming pass: fused accumulate + candidate test + ordered compaction into the row's slot
// (+ top-k: candidate histogram).  One workgroup of kStrNT threads per row, one float4 group per
// thread (short-lived workgroups keep the end of the grid short, where a streaming pass loses
// bandwidth).
// ---------------------------------------------------------------------------------------------
// Threads per workgroup of the streaming selection pass: two float4 groups per thread (a row of
// kTile elements per workgroup).  Measured per pass on ResNet-50 flat, top-k / random-k: 256
// threads (4 groups each) 52.0 / 52.2 us, 512 threads 50.5 / 51.0, 1024 threads 53.1 / 55.8 (one
// barrier across 16 wavefronts holds the whole row back).
constexpr int kStrNT = 512;
constexpr int kStrW = kStrNT / 64;     // its wavefronts

// ZC: some top-k segment of the layout has seg_zc (the form without it has no such test).
template <int KIND, int GDT, bool FUSED, bool ZC = false>
__global__ __launch_bounds__(kStrNT) void k_stream_sel(Tables T, const void* g, const float* src, float* acc_out,
                                                    uint32_t s0, uint32_t s1, uint32_t step, WSel ws) {
  constexpr int kSR = (int)kTile / (4 * kStrNT);  // float4 groups per thread
  __shared__ uint32_t wt[kSR][kStrW];
  __shared__ uint32_t s_hist[KIND == 0 ? kHBins : 1];
  __shared__ uint32_t s_kk[KIND == 1 ? kTile : 1];  // random-k: the candidates' keys, by element
  __shared__ uint32_t wc[kStrW];  // random-k, direct lists: certain winners per wavefront
  __shared__ uint32_t s_und;         // random-k, direct lists: undecided candidates listed so far
  __shared__ uint32_t s_tie[KIND == 0 ? kStrW : 1];  // top-k: elements equal to A per wavefront
  __shared__ uint32_t s_cb;          // the row's first pool entry (a reservation in the overflow pool)
  const uint32_t row = blockIdx.x;
  // the row's segment and bounds: arithmetic on one segment, else one record load (the data loads
  // wait for the bounds only, not for a chain through the segment tables)
  int l = 0;
  uint32_t o = 0, e_ = (uint32_t)T.d, tb = row * kTile;
  uint32_t cb, scap;  // the row's static slot (several segments: loaded with the row's record)
  if (T.L > 1) {
    const uint4 rr = reinterpret_cast<const uint4*>(T.row_rec)[row];
    cb = ws.soff[row];
    scap = ws.soff[row + 1];
    l = (int)rr.x;
    o = rr.y;
    e_ = rr.z;
    tb = rr.w;
    scap -= cb;
  } else {
    static_slot(T, ws, row, cb, scap);
  }
  const uint32_t lo = max(o, tb), hi = min(e_, tb + kTile);
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  uint32_t* R = res_of(ws, l);
  uint32_t mode = 1, A = 0, IA = 0, sh = 0, ulo = 0;
  uint64_t tau = 0;
  const bool direct = KIND == 1 && T.rk_direct;
  bool zc = false;  // top-k, fused: +0 stored at the candidates, not acc
  if constexpr (KIND == 0) {
    mode = R[R_MODE];
    A = R[R_A];
    IA = R[R_IA];
    sh = R[R_SH];
    zc = ZC && FUSED && T.seg_zc[l] != 0u;
  } else {
    tau = T.seg_tau[l];
    ulo = T.seg_ulo[l];
    // the list counter of k_collect starts from zero (this kernel completes before it runs)
    if (!direct && tb == o / kTile * kTile && threadIdx.x < kSubLists) *lcnt_of(ws, l, threadIdx.x) = 0;
  }

  float v[kSR][4];
  uint32_t vm[kSR];
#pragma unroll
  for (int r = 0; r < kSR; ++r) vm[r] = group_mask(tb + (uint32_t)(r * kStrNT + threadIdx.x) * 4u, lo, hi);
  const bool whole = lo == tb && hi == tb + kTile;  // the row is the whole tile (uniform)
  // random-k: the Philox keys of the thread's elements depend on positions only; they are computed
  // while the thread's loads are in flight (called right after the loads are issued)
  uint32_t uk[KIND == 1 ? kSR : 1][4];
  auto random_keys = [&]() {
    if constexpr (KIND == 1) {
#pragma unroll
      for (int r = 0; r < kSR; ++r) {
        const uint32_t i0 = tb + (uint32_t)(r * kStrNT + threadIdx.x) * 4u;
        if ((o & 3u) == 0) {  // the float4 group is one Philox block
          uint4 x = make_uint4(0u, 0u, 0u, 0u);
          if (vm[r]) x = philox(make_uint4((i0 - o) >> 2, 0u, step, kRandkTag | (uint32_t)l), s0, s1);
#pragma unroll
          for (int q = 0; q < 4; ++q) uk[r][q] = word(x, q);
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            uk[r][q] = ((vm[r] >> q) & 1u) ? randk_key(i0 + q - o, (uint32_t)l, step, s0, s1) : 0u;
        }
      }
    }
  };
  if constexpr (FUSED) {
    float gv[kSR][4];
    if (whole) {
#pragma unroll
      for (int r = 0; r < kSR; ++r) {
        const uint32_t i0 = tb + (uint32_t)(r * kStrNT + threadIdx.x) * 4u;
        load4gf<GDT>(g, i0, gv[r]);
        load4f(src, i0, v[r]);
      }
    } else {
#pragma unroll
      for (int r = 0; r < kSR; ++r) {
        const uint32_t i0 = tb + (uint32_t)(r * kStrNT + threadIdx.x) * 4u;
        load4gm<GDT>(g, i0, vm[r], gv[r]);
        load4m(src, i0, vm[r], v[r]);
      }
    }
    random_keys();
#pragma unroll
    for (int r = 0; r < kSR; ++r) {
      const uint32_t i0 = tb + (uint32_t)(r * kStrNT + threadIdx.x) * 4u;
#pragma unroll
      for (int q = 0; q < 4; ++q) v[r][q] = gv[r][q] + v[r][q];
      // top-k: stored at once (+0 at the candidates where seg_zc asks for it: the candidate rule
      // needs only the key); random-k: stored below, once the candidates are known
      if constexpr (KIND == 0) {
        if (zc) {
          float o[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const uint32_t k = mag_key(v[r][q]);
            o[q] = k > A || (mode != 0 && k == A && i0 + q < IA) ? 0.0f : v[r][q];
          }
          store4m(acc_out, i0, vm[r], o);
        } else {
          store4m(acc_out, i0, vm[r], v[r]);
        }
      }
    }
  } else if (KIND == 1 && !src) {
    // random-k without data (a selection prepared ahead of the step): keys and positions only
#pragma unroll
    for (int r = 0; r < kSR; ++r)
#pragma unroll
      for (int q = 0; q < 4; ++q) v[r][q] = 0.0f;
    random_keys();
  } else {
#pragma unroll
    for (int r = 0; r < kSR; ++r) {
      const uint32_t i0 = tb + (uint32_t)(r * kStrNT + threadIdx.x) * 4u;
      if (whole) load4f(src, i0, v[r]);
      else load4m(src, i0, vm[r], v[r]);
    }
    random_keys();
  }
  // candidate flags; wave-level prefixes through ballots, one barrier for the whole row
  uint32_t mask[kSR], lpre[kSR];
  uint32_t kk[kSR][4];
  uint32_t ncert = 0;  // random-k, direct lists: certain winners of this wavefront (uniform)
  uint32_t cbits = 0;  // random-k, direct lists: bit 4r+q marks a certain winner (key below ulo)
  uint32_t ntie = 0;   // top-k, sampled segments: elements equal to A of this wavefront (uniform)
#pragma unroll
  for (int r = 0; r < kSR; ++r) {
    const uint32_t i0 = tb + (uint32_t)(r * kStrNT + threadIdx.x) * 4u;
    uint32_t mk = 0;
    if constexpr (KIND == 0) {
      // sampled segments: keys above A are stored, keys equal to A (the tie bin: exact zeros, say,
      // which may be most of a segment) only counted; exact segments: the winner rule itself
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        kk[r][q] = mag_key(v[r][q]);
        const bool in = (vm[r] >> q) & 1u;
        if (in && (kk[r][q] > A || (mode != 0 && kk[r][q] == A && i0 + q < IA))) mk |= 1u << q;
        if (mode == 0) ntie += (uint32_t)__popcll(__ballot(in && kk[r][q] == A));
      }
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint32_t u = uk[r][q];
        if (((vm[r] >> q) & 1u) && (uint64_t)u < tau) {
          mk |= 1u << q;
          s_kk[(r * kStrNT + threadIdx.x) * 4 + q] = ~u;
        }
        if (((vm[r] >> q) & 1u) && u < ulo) cbits |= 1u << (4 * r + q);
      }
    }
    mask[r] = mk;
    uint32_t pre = 0, tot = 0;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint64_t b = __ballot((mk >> q) & 1u);
      pre += lanes_below(b);
      tot += (uint32_t)__popcll(b);
    }
    lpre[r] = pre;
    if (lane == 0) wt[r][wid] = tot;
    if (direct) {
#pragma unroll
      for (int q = 0; q < 4; ++q) ncert += (uint32_t)__popcll(__ballot((cbits >> (4 * r + q)) & 1u));
    }
  }
  if (direct) {
    if (lane == 0) wc[wid] = ncert;
    if (threadIdx.x == 0) s_und = 0;
  }
  if constexpr (KIND == 0) {
    if (lane == 0) s_tie[wid] = ntie;
  }
  if constexpr (FUSED && KIND == 1) {
    // random-k (as top-k segments with seg_zc, above): the residual is stored as +0 at every
    // candidate; the emit kernel puts the value back at the few candidates that do not win (the
    // window's losers, about 6 sqrt(k_l) + 32 of a segment), and the exact path puts them all back
    // first.  Zeroing the winners afterwards instead wrote single words into lines long evicted
    // from the caches: 1e9 elements at 10 %, 1.9 of the emission's 2.3 ms.
#pragma unroll
    for (int r = 0; r < kSR; ++r) {
      const uint32_t i0 = tb + (uint32_t)(r * kStrNT + threadIdx.x) * 4u;
      float o[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) o[q] = ((mask[r] >> q) & 1u) ? 0.0f : v[r][q];
      store4m(acc_out, i0, vm[r], o);
    }
  }
  __syncthreads();
  // the row's candidates go to its static slot, or, when there are more than it holds, to entries
  // reserved in the overflow pool; a row that does not fit is dropped and its segment takes the
  // exact path (the histogram still counts its candidates)
  // (the wavefront totals are read once: the row's total, and each group's first position for
  // this wavefront; the total and the slot are uniform, kept in scalar registers)
  uint32_t tot = 0, rbs[kSR];
#pragma unroll
  for (int r = 0; r < kSR; ++r) {
    uint32_t pre = 0, all = 0;
#pragma unroll
    for (int w = 0; w < kStrW; ++w) {
      const uint32_t c = wt[r][w];
      pre += w < wid ? c : 0u;
      all += c;
    }
    rbs[r] = tot + pre;
    tot += all;
  }
  tot = __builtin_amdgcn_readfirstlane(tot);
  if (tot > scap) {
    if (threadIdx.x == 0) s_cb = pool_reserve(ws, row, tot);
    __syncthreads();
    cb = __builtin_amdgcn_readfirstlane(s_cb);
  }
  const bool dropped = cb == kDropped;
  if (threadIdx.x == 0 && (T.L > 1 || tot > scap)) ws.coff[row] = cb;
  if (dropped) {
    if constexpr (KIND == 0) {
      if (threadIdx.x == 0) atomicOr(&R[R_OVF], 1u);
    }
    if (FUSED && (KIND == 1 || zc)) {
      // the candidates' values were stored as +0 above; without the candidates the exact path
      // cannot restore them, so they are stored again now
#pragma unroll
      for (int r = 0; r < kSR; ++r) {
        const uint32_t i0 = tb + (uint32_t)(r * kStrNT + threadIdx.x) * 4u;
        store4m(acc_out, i0, vm[r], v[r]);
      }
    }
  }
  uint32_t* cidx = ws.cand_idx + cb;
  float* cval = ws.cand_val + cb;
  uint32_t* ckey = ws.cand_key + cb;
#pragma unroll
  for (int r = 0; r < kSR; ++r) {
    if (mask[r] && !dropped) {
      const uint32_t i0 = tb + (uint32_t)(r * kStrNT + threadIdx.x) * 4u;
      uint32_t pos = rbs[r] + lpre[r];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if ((mask[r] >> q) & 1u) {
          uint32_t key;
          if constexpr (KIND == 0) key = kk[r][q];
          else key = s_kk[(r * kStrNT + threadIdx.x) * 4 + q];
          cidx[pos] = i0 + q;
          cval[pos] = v[r][q];
          ckey[pos] = key;
          ++pos;
          if (direct && !((cbits >> (4 * r + q)) & 1u)) {
            // random-k, direct lists: an undecided candidate ([ulo, tau)) joins the row's list as
            // a (key', index) pair, at the row's pool entries in the pair array (fewer than its
            // candidates)
            const uint32_t p = atomicAdd(&s_und, 1u);
            ws.pairs[(size_t)cb + p] = make_uint2(key, i0 + q);
          }
        }
      }
    }
  }
  const uint32_t base = tot;  // the row's candidates
  if (threadIdx.x == 0) ws.counts[row] = base;
  if (direct && threadIdx.x == 0) {
    // random-k, direct lists: the row's certain winners (key below ulo)
    uint32_t c = 0;
#pragma unroll
    for (int w = 0; w < kStrW; ++w) c += wc[w];
    ws.rcnt[row] = c;
  }
  if constexpr (KIND == 0) {
    if (mode == 0 && threadIdx.x == 0) {
      // the ties are the histogram's bin 0
      uint32_t t = 0;
#pragma unroll
      for (int w = 0; w < kStrW; ++w) t += s_tie[w];
      ws.rtie[row] = t;
      if (t) atomicAdd(&ws.hist[((size_t)l * kHCopies + (row % kHCopies)) * kHBins], t);
    }
    if (mode == 0 && base) {
      uint32_t* gh = ws.hist + ((size_t)l * kHCopies + (row % kHCopies)) * kHBins;
      if (base > kHistDirect) {  // many candidates: count them in LDS, then one atomic per used bin
        for (int b = threadIdx.x; b < kHBins; b += kStrNT) s_hist[b] = 0;
        __syncthreads();
#pragma unroll
        for (int r = 0; r < kSR; ++r)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if ((mask[r] >> q) & 1u) atomicAdd(&s_hist[cand_bin(kk[r][q], A, sh)], 1u);
        __syncthreads();
        for (int b = threadIdx.x; b < kHBins; b += kStrNT) {
          const uint32_t c = s_hist[b];
          if (c) atomicAdd(&gh[b], c);
        }
      } else {
#pragma unroll
        for (int r = 0; r < kSR; ++r)
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if ((mask[r] >> q) & 1u) atomicAdd(&gh[cand_bin(kk[r][q], A, sh)], 1u);
      }
    }
  }
}

// Top-k, per segment: the histogram bin B holding the k_l-th best candidate and how many winners
// it still has to give; fewer than k_l candidates in all marks the segment for the exact path.
__global__ __launch_bounds__(kSelNT) void k_resolve(Tables T, WSel ws0, Batch BT) {
  const WSel ws = ws_at(ws0, (uint64_t)blockIdx.y * BT.ws);
  __shared__ uint32_t hist[kHBins];
  __shared__ uint32_t lds[2 * kSelNT / 64];
  const int l = blockIdx.x;
  uint32_t* R = res_of(ws, l);
  // the segment's mode and every copy of its histogram in one round trip (a segment of mode 1 has
  // no histogram: its loads read the unused copies and are dropped)
  constexpr int kPer = kHBins / kSelNT;
  static_assert(kHBins % kSelNT == 0, "whole bins per thread");
  const uint32_t mode = R[R_MODE], ovf = R[R_OVF];
  const uint32_t* gh = ws.hist + (size_t)l * kHCopies * kHBins;
  uint32_t c[kPer][kHCopies];
#pragma unroll
  for (int u = 0; u < kPer; ++u)
#pragma unroll
    for (int x = 0; x < kHCopies; ++x) c[u][x] = gh[x * kHBins + u * kSelNT + threadIdx.x];
  if (mode != 0) return;
#pragma unroll
  for (int u = 0; u < kPer; ++u) {
    uint32_t sum = 0;
#pragma unroll
    for (int x = 0; x < kHCopies; ++x) sum += c[u][x];
    hist[u * kSelNT + threadIdx.x] = sum;
  }
  __syncthreads();
  const uint32_t kl = (uint32_t)T.seg_k[l];
  uint32_t above;
  const int bin = block_resolve<kSelNT>(hist, kHBins, kl, lds, above);
  if (threadIdx.x < kSubLists) *lcnt_of(ws, l, threadIdx.x) = 0;
  if (ovf) {
    // A row's candidates did not fit the workspace (the sample put A far below the k_l-th key), but
    // the histogram counted them all: the rows collect again the keys of bins >= B only (those
    // above bin B are certain, bin B's are listed), as a retry (below) does.  With one segment the
    // pool's parts start again from empty (every row is collected again), unless the pass stored
    // +0 at the candidates: the rows then read their old candidates to put them back into acc, so
    // those must stay where they are.  The threshold bin being the key A itself, or the retry
    // switched off: the exact path.
    const uint32_t A = R[R_A], sh = R[R_SH];
    if (bin < 1 || !T.tk_retry) {
      if (threadIdx.x == 0) {
        R[R_SLOW] = 1;
        R[R_RETRY] = 0;
        atomicOr(ws.diag, kDiagSlowPath);
      }
      return;
    }
    if (T.L == 1 && !T.seg_zc[l] && threadIdx.x < (unsigned)kPools) *pcnt_of(ws, threadIdx.x) = 0u;
    if (threadIdx.x == 0) {
      const uint32_t b = (uint32_t)bin;
      R[R_A2] = A + ((b - 1u) << sh);  // keys above it: bins >= B
      R[R_A] = b < (uint32_t)kHBins - 1u ? A + 1u + (b << sh) : 0xFFFFFFFFu;  // first key of bin B + 1
      R[R_NEED] = kl - above;
      R[R_B] = 1u;  // not the tie bin: the listed candidates are ranked
      R[R_RETRY] = 1u;
      R[R_OVF] = 0u;
      atomicOr(ws.diag, kDiagRetry);
    }
    return;
  }
  if (bin >= 0) {
    if (threadIdx.x == 0) {
      R[R_B] = (uint32_t)bin;
      R[R_NEED] = kl - above;
      R[R_RETRY] = 0;
    }
    return;
  }
  // Fewer than k_l candidates: the sample misjudged the density above A.  The retry threshold A2
  // is read from the same sample, at the rank where the density actually found (N keys above A
  // against s sampled ones) predicts 4 k_l + 256 keys above it; its rows then collect every key
  // above A2 again and count those equal to it (k_collect), and k_select falls back to the exact
  // whole-segment path only if those are still fewer than k_l.
  uint32_t mine = 0;
#pragma unroll
  for (int u = 0; u < kPer; ++u) mine += hist[u * kSelNT + threadIdx.x];
  uint32_t N;
  (void)block_excl_scan<kSelNT>(mine, lds, N);
  const uint32_t A = R[R_A];
  const uint32_t ns = ((uint32_t)T.seg_ro[l + 1] - (uint32_t)T.seg_ro[l]) * kSampleRun;
  const uint32_t* sk = ws.samp + (size_t)T.seg_ro[l] * kSampleRun;
  __syncthreads();
  for (int b = threadIdx.x; b < kHBins; b += kSelNT) hist[b] = 0;
  __syncthreads();
  uint32_t above_a = 0;
  for_keys(sk, ns, [&](uint32_t, uint32_t k) {
    atomicAdd(&hist[k >> 20], 1u);
    above_a += k >= A ? 1u : 0u;
  });
  uint32_t sA;
  (void)block_excl_scan<kSelNT>(above_a, lds, sA);  // its barriers also publish hist
  // (at least the rank where the sample alone predicts 4 k_l + 64 keys, in case its top was the
  // only part it misjudged; only that rank when fewer than 8 sampled keys reach A: the scale
  // N / s is then too noisy to use, and too large a threshold would overflow the candidate pool)
  const uint32_t n_seg = (uint32_t)T.seg_off[l + 1] - (uint32_t)T.seg_off[l];
  const uint64_t plain = (((uint64_t)4 * kl + 64u) * ns + n_seg - 1u) / n_seg;
  const uint64_t want = sA >= 8u ? ((uint64_t)4 * kl + 256u) * (uint64_t)sA : 0u;
  const uint64_t ratio = (want + max(N, 1u) - 1u) / max(N, 1u);
  const uint32_t r2 = (uint32_t)min<uint64_t>((uint64_t)ns, max(plain, ratio));
  uint32_t a2above;
  const int b2 = block_resolve<kSelNT>(hist, kHBins, r2, lds, a2above);
  const uint32_t A2 = b2 < 0 || r2 >= ns ? 0u : min(A, (uint32_t)b2 << 20);
  if (threadIdx.x == 0) {
    if (!T.tk_retry || A2 >= A) {
      R[R_SLOW] = 1;
      R[R_RETRY] = 0;
      atomicOr(ws.diag, kDiagSlowPath);
    } else {
      R[R_RETRY] = 1u;
      R[R_A2] = A2;
      R[R_NEED] = kl - N;
      R[R_B] = 1u;  // not the tie bin: the listed candidates are ranked
      atomicOr(ws.diag, kDiagRetry);
    }
  }
}

// Per row: candidates certain to win are counted; the undecided ones go to the segment's list (in
// any order: the selection over the list does not depend on it; row r appends to sub-list
// r % kSubLists, which spreads the atomics on the list counters).  Top-k: above / inside bin B of
// a histogrammed segment.  Random-k: Philox key below ulo_l / in [ulo_l, tau_l).
// One wavefront per CR consecutive rows (CR = 1 for one or a few workers, where the rows are the
// whole grid; more per wavefront for a batch): the rows' segments, candidate counts and first 64
// candidate keys are loaded together; counts and list positions come from ballots, and each chunk
// of 64 candidates reserves its list space with one atomic.
// Top-k candidate retry, one wavefront per row: the row's keys are read again from acc and every
// key > A2 becomes a candidate, in index order, in the row's static slot or, if more, in entries
// reserved in the overflow pool; those >= A (the first candidates) are certain winners, those in
// (A2, A) go to the segment's list, and the keys equal to A2 are counted (ties, taken by index if
// the list falls short).  A row or a list that does not fit marks the segment for the exact path.
__device__ __forceinline__ void collect_retry(const Tables& T, const WSel& ws, const Batch& BT, uint32_t row, int l,
                                              uint32_t* R) {
  const uint32_t lane = threadIdx.x & 63;
  const float* acc = BT.g[blockIdx.y] ? BT.e[blockIdx.y] : BT.src[blockIdx.y];
  uint32_t o = 0, e_ = (uint32_t)T.d, tb = row * kTile;
  if (T.L > 1) {
    const uint4 rr = reinterpret_cast<const uint4*>(T.row_rec)[row];
    o = rr.y;
    e_ = rr.z;
    tb = rr.w;
  }
  const uint32_t lo = max(o, tb), hi = min(e_, tb + kTile);
  const uint32_t A = R[R_A], A2 = R[R_A2];
  const uint32_t r0 = (uint32_t)T.seg_cbase[l], c = (row - r0) % kSubLists, lq = T.seg_lq[l];
  const size_t sb = sublist_base(T, l, c);
  if (BT.g[blockIdx.y] && T.seg_zc[l]) {
    // the pass stored +0 at the row's candidates: their values go back into acc first (a dropped
    // row's pass stored acc itself), made visible to this wavefront's reads below
    float* accw = BT.e[blockIdx.y];
    const uint32_t oc = ws.counts[row];
    const uint32_t oco = row_entry(T, ws, row, oc, ws.coff[row]);
    if (oco != kDropped)
      for (uint32_t j = lane; j < oc; j += 64) accw[ws.cand_idx[(size_t)oco + j]] = ws.cand_val[(size_t)oco + j];
    __threadfence();
  }
  // pass 1: how many (above A2, and equal)
  uint32_t n = 0, nt = 0;
  for (uint32_t i0 = lo; i0 < hi; i0 += 64) {
    const uint32_t i = i0 + lane;
    const uint32_t k = i < hi ? mag_key(acc[i]) : 0u;
    n += (uint32_t)__popcll(__ballot(i < hi && k > A2));
    nt += (uint32_t)__popcll(__ballot(i < hi && k == A2));
  }
  if (lane == 0) ws.rtie[row] = nt;
  uint32_t cb, scap;
  static_slot(T, ws, row, cb, scap);
  if (n > scap) {
    uint32_t at = 0;
    if (lane == 0) at = pool_reserve(ws, row, n);
    cb = __shfl(at, 0, 64);
  }
  if (lane == 0) ws.coff[row] = cb;
  if (cb == kDropped) {
    if (lane == 0) atomicOr(&R[R_OVF], 1u);
    return;
  }
  // pass 2: the candidates and the list
  uint32_t* cidx = ws.cand_idx + cb;
  float* cval = ws.cand_val + cb;
  uint32_t* ckey = ws.cand_key + cb;
  uint32_t m = 0, na = 0;
  for (uint32_t i0 = lo; i0 < hi; i0 += 64) {
    const uint32_t i = i0 + lane;
    const float v = i < hi ? acc[i] : 0.0f;
    const uint32_t key = mag_key(v);
    const bool take = i < hi && key > A2, cert = take && key >= A, lst = take && !cert;
    const uint64_t bt = __ballot(take), bl = __ballot(lst);
    if (take) {
      const uint32_t pos = m + lanes_below(bt);
      cidx[pos] = i;
      cval[pos] = v;
      ckey[pos] = key;
    }
    m += (uint32_t)__popcll(bt);
    na += (uint32_t)__popcll(__ballot(cert));
    const uint32_t nl = (uint32_t)__popcll(bl);
    if (nl) {
      uint32_t base = 0;
      if (lane == 0) base = atomicAdd(lcnt_of(ws, l, c), nl);
      base = __shfl(base, 0, 64);
      const uint32_t t = base + lanes_below(bl);
      if (lst && t < lq) {  // a full sub-list is seen by k_select (its count exceeds lq)
        const size_t p = sb + t;
        ws.list_key[p] = key;
        ws.list_idx[p] = i;
      }
    }
  }
  if (lane == 0) {
    ws.counts[row] = m;
    ws.rcnt[row] = na;
  }
}

constexpr uint32_t kCollectBuf = 512;  // listed candidates a wavefront of k_collect stages in LDS

template <int KIND, uint32_t kCollectRows>
__global__ __launch_bounds__(kNT) void k_collect(Tables T, WSel ws0, Batch BT) {
  const WSel ws = ws_at(ws0, (uint64_t)blockIdx.y * BT.ws);
  __shared__ uint32_t s_lk[kNT / 64][kCollectBuf], s_li[kNT / 64][kCollectBuf];
  const uint32_t lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const uint32_t row0 = (blockIdx.x * (kNT / 64) + (threadIdx.x >> 6)) * kCollectRows;
  int ls[kCollectRows];
  uint32_t cnts[kCollectRows], cofs[kCollectRows], k0[kCollectRows], i0[kCollectRows];
  // one segment: its record read once, in the first round trip (k_collect does not write it; read
  // per row, each row's fields waited for again after the previous row's list stores)
  uint32_t r_skip = 0, r_retry = 0, r_A = 0, r_sh = 0, r_B = 0;
  if (KIND == 0 && T.L == 1) {
    const uint32_t* R0 = res_of(ws, 0);
    r_skip = R0[R_SLOW] | R0[R_MODE];
    r_retry = R0[R_RETRY];
    r_A = R0[R_A];
    r_sh = R0[R_SH];
    r_B = R0[R_B];
  }
#pragma unroll
  for (uint32_t r = 0; r < kCollectRows; ++r) {
    const uint32_t row = min(row0 + r, (uint32_t)T.nrows - 1u);
    ls[r] = T.L == 1 ? 0 : T.row_seg[row];  // one segment: no load before the segment's record
    cnts[r] = ws.counts[row];
    cofs[r] = ws.coff[row];
    // one segment: the first 64 keys and indices from the row's static slot, in the same round
    // trip (used if the row's candidates are there; past the count: unused, and not loaded past
    // the slot)
    const uint32_t cap0 = min(ws.S, (uint32_t)T.d - row * kTile);
    const bool in0 = T.L == 1 && lane < cap0;
    k0[r] = in0 ? ws.cand_key[(size_t)row * ws.S + lane] : 0u;
    i0[r] = in0 ? ws.cand_idx[(size_t)row * ws.S + lane] : 0u;
  }
#pragma unroll
  for (uint32_t r = 0; r < kCollectRows; ++r) {
    const uint32_t row = row0 + r;
    if (row >= (uint32_t)T.nrows) break;
    const int l = ls[r];
    uint32_t* R = res_of(ws, l);
    uint32_t A = 0, sh = 0, B = 0, ulo = 0;
    if constexpr (KIND == 0) {
      const bool one = T.L == 1;
      if (one ? r_skip != 0 : (R[R_SLOW] || R[R_MODE])) continue;
      if (one ? r_retry != 0 : R[R_RETRY] != 0) {
        collect_retry(T, ws, BT, row, l, R);
        continue;
      }
      A = one ? r_A : R[R_A];
      sh = one ? r_sh : R[R_SH];
      B = one ? r_B : R[R_B];
    } else {
      ulo = T.seg_ulo[l];
    }
    const uint32_t co = row_entry(T, ws, row, cnts[r], cofs[r]);
    if (co == kDropped) continue;  // the segment takes the exact path
    // class: 2 = certain winner, 1 = undecided (listed), 0 = loses
    auto cls = [&](uint32_t k) -> uint32_t {
      if constexpr (KIND == 0) {
        const uint32_t b = cand_bin(k, A, sh);
        return b > B ? 2u : (b == B ? 1u : 0u);
      } else {
        return ~k < ulo ? 2u : 1u;
      }
    };
    // tie bin (the threshold bin is the key A alone, whose elements the pass only counted): every
    // stored candidate is a certain winner and nothing is listed
    const bool tie_bin = KIND == 0 && B == 0;
    const uint32_t cnt = cnts[r];
    const uint32_t* ck = ws.cand_key + co;
    const uint32_t* ci = ws.cand_idx + co;
    const bool k0_ok = T.L == 1 && co == row * ws.S;
    const uint32_t r0 = (uint32_t)T.seg_cbase[l], c = (row - r0) % kSubLists, lq = T.seg_lq[l];
    const size_t sb = sublist_base(T, l, c);
    // The row's listed candidates are staged in the wavefront's LDS buffer and written out with
    // one reservation of list space per row (or per full buffer).  An atomic per chunk of 64
    // candidates, each waited for, on the 16 sub-list counters took 92-141 us to collect BERT flat
    // at 10 % with bf16 values (211,000 equal keys in the threshold bin); staged, 30 us.
    uint32_t na = 0, nb = 0;  // certain winners; listed candidates in the buffer (uniform)
    auto flush = [&]() {
      uint32_t base = 0;
      if (lane == 0) base = atomicAdd(lcnt_of(ws, l, c), nb);
      base = __shfl(base, 0, 64);
      for (uint32_t x = lane; x < nb; x += 64) {
        const uint32_t t = base + x;
        if (t < lq) {  // a full sub-list is seen by k_select (its count exceeds lq)
          ws.list_key[sb + t] = s_lk[wv][x];
          ws.list_idx[sb + t] = s_li[wv][x];
        }
      }
      nb = 0;
    };
    uint32_t kc = k0_ok ? k0[r] : (lane < cnt ? ck[lane] : 0u);
    for (uint32_t j0 = 0; j0 < cnt; j0 += 64) {
      const uint32_t j = j0 + lane;
      const uint32_t k = kc;
      if (j0 + 64 < cnt) kc = j + 64 < cnt ? ck[j + 64] : 0u;  // the next chunk's keys, in flight
      const uint32_t cl = j < cnt ? (tie_bin ? 2u : cls(k)) : 0u;
      na += (uint32_t)__popcll(__ballot(cl == 2u));
      const uint64_t bu = __ballot(cl == 1u);
      const uint32_t nu = (uint32_t)__popcll(bu);
      if (nu == 0) continue;
      if (nb + nu > kCollectBuf) flush();
      if (cl == 1u) {
        const uint32_t x = nb + lanes_below(bu);
        s_lk[wv][x] = k;
        s_li[wv][x] = k0_ok && j0 == 0 ? i0[r] : ci[j];
      }
      nb += nu;
    }
    if (nb) flush();
    if (lane == 0) ws.rcnt[row] = na;
  }
}

// An entry to be ranked as one 64-bit word: key' in the high half and the complement of the index
// in the low half, so that one unsigned comparison orders entries by key' descending, then index
// ascending.  The word 0 (key' 0 with index 2^32 - 1, which no element has) beats no entry; it
// pads a ranked list to rank_pad(m) words, the stride of the ranking loop.
__device__ __forceinline__ uint64_t rank_word(uint32_t key, uint32_t idx) {
  return ((uint64_t)key << 32) | (uint64_t)(~idx);
}
__device__ __forceinline__ uint32_t rank_pad(uint32_t m) { return (m + 63u) & ~63u; }

// The need-th best (1 <= need <= m <= kRankList) of m entries held in LDS as rank words, padded
// with zero words up to rank_pad(m): every entry counts the entries that beat it.  An entry is
// shared by 4, 8 or 16 threads (as many as the workgroup's threads allow for m entries), each
// comparing against every 4th, 8th or 16th entry, four loads in flight per pass.  Gives its key'
// and one past its index.
__device__ __forceinline__ void rank_select(const uint64_t* g, uint32_t m, uint32_t need, uint32_t& T_out,
                                            uint32_t& IT_out) {
  static_assert(kRankList * 4 <= kSelNT, "four threads per ranked entry");
  __shared__ uint32_t s_t, s_it;
  const uint32_t lg = m <= kSelNT / 16 ? 4u : (m <= kSelNT / 8 ? 3u : 2u);  // log2 threads per entry
  const uint32_t tpe = 1u << lg;
  const uint32_t e = threadIdx.x >> lg, part = threadIdx.x & (tpe - 1u);
  uint32_t rank = 0;
  uint64_t v = 0;
  if (e < m) {
    v = g[e];
    // j0 + 3 tpe stays below m rounded up to 4 tpe, which divides 64: inside the padding
    for (uint32_t j0 = part; j0 < m; j0 += 4u * tpe) {
      uint64_t w[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) w[u] = g[j0 + (uint32_t)u * tpe];
#pragma unroll
      for (int u = 0; u < 4; ++u) rank += w[u] > v ? 1u : 0u;
    }
  }
  // the entry's threads are adjacent lanes of one wavefront
  rank += __shfl_xor(rank, 1, 64);
  rank += __shfl_xor(rank, 2, 64);
  if (lg >= 3u) rank += __shfl_xor(rank, 4, 64);
  if (lg >= 4u) rank += __shfl_xor(rank, 8, 64);
  if (e < m && part == 0 && rank == need - 1) {
    s_t = (uint32_t)(v >> 32);
    s_it = ~(uint32_t)v + 1u;
  }
  __syncthreads();
  T_out = s_t;
  IT_out = s_it;
  __syncthreads();
}

// The need best of the m listed candidates (key' descending, then index ascending; 1 <= need <=
// m): the key' T of the last winner and one past its index (every listed winner is key' > T, or
// key' == T with index below that bound).  Radix levels of 11 bits narrow the key' range until
// the bin holding the need-th best has at most kRankList entries; those are gathered and ranked.
// kand / kor: the AND and the OR of the m keys (needed when m > kRankList).
template <typename K, typename I>
__device__ __forceinline__ void list_threshold_ao(const K& key, const I& idx, uint32_t m, uint32_t need,
                                                  uint32_t kand, uint32_t kor, uint32_t* hist, uint32_t* lds,
                                                  uint64_t* g, uint32_t& T_out, uint32_t& IT_out,
                                                  uint32_t* defer_need) {
  __shared__ uint32_t s_n;
  if (m <= kRankList) {
    for (uint32_t j = threadIdx.x; j < rank_pad(m); j += kSelNT) g[j] = j < m ? rank_word(key[j], idx[j]) : 0ull;
    __syncthreads();
    rank_select(g, m, need, T_out, IT_out);
    return;
  }
  const uint32_t diff = kand ^ kor;
  uint32_t prefix = kand, known = 32;  // all keys equal: nothing to resolve
  uint32_t cnt = m;
  if (diff) {
    const int h = 31 - __clz(diff);
    prefix = h == 31 ? 0u : (kand & (0xFFFFFFFFu << (h + 1)));
    known = (uint32_t)(31 - h);
    while (known < 32 && cnt > kRankList) {
      const int w = min(11, 32 - (int)known);
      const int shift = 32 - (int)known - w;
      for (int b = threadIdx.x; b < (1 << w); b += kSelNT) hist[b] = 0;
      __syncthreads();
      const uint32_t pmask = known == 0 ? 0u : (0xFFFFFFFFu << (32 - known));
      const uint32_t want = prefix & pmask;
      for_keys(key, m, [&](uint32_t, uint32_t k) {
        if ((k & pmask) == want) atomicAdd(&hist[(k >> shift) & ((1u << w) - 1u)], 1u);
      });
      __syncthreads();
      uint32_t above;
      const int bin = block_resolve<kSelNT>(hist, 1 << w, need, lds, above);
      cnt = hist[max(bin, 0)];
      __syncthreads();
      prefix |= (uint32_t)max(bin, 0) << shift;
      need -= above;
      known += (uint32_t)w;
    }
  }
  if (cnt <= kRankList) {  // gather the entries sharing the resolved prefix and rank them
    const uint32_t pmask = known == 0 ? 0u : (known >= 32 ? 0xFFFFFFFFu : (0xFFFFFFFFu << (32 - known)));
    const uint32_t want = prefix & pmask;
    if (threadIdx.x == 0) s_n = 0;
    for (uint32_t j = cnt + threadIdx.x; j < rank_pad(cnt); j += kSelNT) g[j] = 0ull;  // the gather fills [0, cnt)
    __syncthreads();
    for_keys(key, m, [&](uint32_t f, uint32_t k) {
      if ((k & pmask) == want) {
        const uint32_t p = atomicAdd(&s_n, 1u);
        g[p] = rank_word(k, idx[f]);
      }
    });
    __syncthreads();
    rank_select(g, cnt, need, T_out, IT_out);
    return;
  }
  // more than kRankList entries share the full key': ties ordered by index (with defer_need, the
  // caller resolves them: IT_out = kTieRows, *defer_need = how many of them win)
  T_out = prefix;
  if (need >= cnt) {
    IT_out = 0xFFFFFFFFu;
  } else if (defer_need) {
    IT_out = kTieRows;
    *defer_need = need;
  } else {
    IT_out = block_nth_smallest_tie(key, idx, m, prefix, need, hist, lds) + 1u;
  }
}

template <typename K>
__device__ __forceinline__ void list_threshold(const K& key, const K& idx, uint32_t m, uint32_t need,
                                               uint32_t* hist, uint32_t* lds, uint64_t* g,
                                               uint32_t& T_out, uint32_t& IT_out, uint32_t* defer_need = nullptr) {
  uint32_t kand = 0xFFFFFFFFu, kor = 0u;
  if (m > kRankList) {
    for_keys(key, m, [&](uint32_t, uint32_t k) {
      kand &= k;
      kor |= k;
    });
    block_and_or(kand, kor, lds);
  }
  list_threshold_ao(key, idx, m, need, kand, kor, hist, lds, g, T_out, IT_out, defer_need);
}

// Per segment: the exact threshold among the listed candidates, then every row's message offset;
// or the exact whole-segment path when the candidates cannot hold the answer.  Independent loads
// are issued together (record, sub-list sizes, the rows' counts) to keep the chain of dependent
// memory round trips short.  BIG (layouts with a very large k_l): only the threshold; the rows'
// winners are then counted by k_rowcount and scanned by k_rowscan, both spread over many
// workgroups, instead of one workgroup adding the list's winners to their rows.
template <int KIND, bool BIG>
__global__ __launch_bounds__(kSelNT) void k_select(Tables T, WSel ws0, uint32_t* out_idx, float* out_val,
                                                   uint32_t step, Batch BT) {
  const WSel ws = ws_at(ws0, (uint64_t)blockIdx.y * BT.ws);
  float* e_zero = BT.e[blockIdx.y];
  const float* data = BT.g[blockIdx.y] ? BT.e[blockIdx.y] : BT.src[blockIdx.y];  // acc
  out_idx = shifted(out_idx, (uint64_t)blockIdx.y * BT.msg * 4u);
  out_val = out_val ? shifted(out_val, (uint64_t)blockIdx.y * BT.msg * 4u) : nullptr;
  const uint32_t s0 = BT.seed_lo[blockIdx.y], s1 = BT.seed_hi[blockIdx.y];
  constexpr uint32_t kPer = kSelPer;  // rows per thread held in registers (more are re-read)
  __shared__ uint32_t hist[kHBins];
  __shared__ uint32_t lds[3 * kSelNT / 64];
  __shared__ uint32_t s_key[kListLds];
  __shared__ uint32_t s_idx[kListLds];
  __shared__ uint32_t s_add[kRowsLds];
  __shared__ uint64_t s_g[kRankList];
  const int l = blockIdx.x;
  uint32_t* R = res_of(ws, l);
  // (one segment: no table loads before the rows' loads)
  const uint32_t r0 = T.L == 1 ? 0u : (uint32_t)T.seg_cbase[l];
  const uint32_t nr = T.L == 1 ? (uint32_t)T.nrows : (uint32_t)T.seg_cbase[l + 1] - r0;
  const uint32_t kl = T.L == 1 ? (uint32_t)T.K : (uint32_t)T.seg_k[l];
  const uint32_t per = (nr + kSelNT - 1) / kSelNT;
  const uint32_t a = min(nr, threadIdx.x * per), b = min(nr, a + per);
  const uint32_t* rc = ws.rcnt + r0;
  const uint32_t* cc = ws.counts + r0;
  // round trip 1: record, sub-list sizes, row counts
  bool slow = false, listed = true;
  uint32_t need = 0, mU = 0, exU = 0, ovf = 0;
  if constexpr (KIND == 0) {
    slow = R[R_SLOW] != 0;
    listed = R[R_MODE] == 0;
    need = R[R_NEED];
    ovf = R[R_OVF];
  }
  const bool direct = KIND == 1 && T.rk_direct;
  const uint32_t lq = T.seg_lq[l];
  uint32_t lc[kSubLists];
#pragma unroll
  for (int c = 0; c < kSubLists; ++c) lc[c] = direct ? 0u : *lcnt_of(ws, l, (uint32_t)c);
  bool lfull = false;  // a sub-list overflowed its region
#pragma unroll
  for (int c = 0; c < kSubLists; ++c) lfull |= lc[c] > lq;
  // top-k candidate retry whose list holds fewer than the `need` winners: every listed candidate
  // wins, and the rest are the first elements equal to A2 (counted per row, not stored)
  bool retry_ties = false;
  if constexpr (KIND == 0) {
    // a row or a sub-list that did not fit the workspace: the exact path
    if (!slow) {
      uint32_t m = 0;
#pragma unroll
      for (int c = 0; c < kSubLists; ++c) m += lc[c];
      retry_ties = listed && R[R_RETRY] && m < need;
      if (retry_ties) need -= m;
      if (ovf || (listed && lfull)) {
        slow = true;
        __syncthreads();  // every thread has read R_SLOW before it is set
        if (threadIdx.x == 0) {
          R[R_SLOW] = 1u;
          atomicOr(ws.diag, kDiagSlowPath);
        }
      }
    }
  }
  // random-k on a layout with very many rows needs only the totals: the rows are summed with
  // coalesced strided loads there, not in per-thread runs (one workgroup reading 244,141 rows in
  // runs of 238 per thread took 0.44 ms at 1e9 elements)
  const bool strided = KIND == 1 && !direct && BIG;
  // random-k: the rows' first pool entries (one segment: the static slot, r * S, unless the row
  // holds more candidates than it, so only those rows' entries are loaded)
  const uint32_t* ro = ws.coff + r0;
  auto first_entry = [&](uint32_t x, uint32_t cnt) -> uint32_t {
    const uint32_t row = r0 + x;
    return cnt > min(ws.S, (uint32_t)T.d - row * kTile) ? ro[x] : row * ws.S;
  };
  uint32_t cr[kPer], cn[kPer], co[kPer];
#pragma unroll
  for (uint32_t x = 0; x < kPer; ++x) {
    cr[x] = !strided && a + x < b ? rc[a + x] : 0u;
    cn[x] = !strided && a + x < b ? cc[a + x] : 0u;
    co[x] = KIND == 1 && T.L > 1 && !strided && a + x < b ? ro[a + x] : 0u;
  }
  if (KIND == 1 && T.L == 1 && !strided) {
#pragma unroll
    for (uint32_t x = 0; x < kPer; ++x)
      if (a + x < b) co[x] = first_entry(a + x, cn[x]);
  }
  if constexpr (KIND == 1) {
    // random-k: the certain winners S (keys below ulo) and the candidates N decide whether the
    // window [ulo, tau) holds the k_l-th smallest key (also counted: rows whose candidates did not
    // fit the workspace)
    uint32_t sv[3] = {0u, 0u, 0u};
    if (strided) {
      constexpr uint32_t kU = 8;
      for (uint32_t x0 = threadIdx.x; x0 < nr; x0 += kU * kSelNT) {
        uint32_t ra[kU], ca[kU], oa[kU];
#pragma unroll
        for (uint32_t u = 0; u < kU; ++u) {
          const uint32_t x = x0 + u * kSelNT;
          ra[u] = x < nr ? rc[x] : 0u;
          ca[u] = x < nr ? cc[x] : 0u;
          oa[u] = x < nr && T.L > 1 ? ro[x] : 0u;
        }
#pragma unroll
        for (uint32_t u = 0; u < kU; ++u) {
          const uint32_t x = x0 + u * kSelNT;
          if (T.L == 1 && x < nr) oa[u] = first_entry(x, ca[u]);
          sv[0] += ra[u];
          sv[1] += ca[u];
          sv[2] += oa[u] == kDropped ? 1u : 0u;
        }
      }
    } else {
#pragma unroll
      for (uint32_t x = 0; x < kPer; ++x) {
        sv[0] += cr[x];
        sv[1] += cn[x];
        sv[2] += co[x] == kDropped ? 1u : 0u;
      }
      for (uint32_t x = a + kPer; x < b; ++x) {
        const uint32_t c = cc[x];
        sv[0] += rc[x];
        sv[1] += c;
        sv[2] += (T.L == 1 ? first_entry(x, c) : ro[x]) == kDropped ? 1u : 0u;
      }
    }
    uint32_t ex[3], tot[3];
    block_excl_scan_n<kSelNT, 3>(sv, lds, ex, tot);
    const uint32_t S = tot[0], N = tot[1];
    // direct lists: the rows' undecided candidates (counts - certain) must fit the LDS list;
    // collected lists: every sub-list its region
    slow = S > kl || N < kl || tot[2] != 0 || (direct ? N - S > kListLds : lfull);
    need = kl - S;
    mU = N - S;
    exU = ex[1] - ex[0];
    if (threadIdx.x == 0) {
      R[R_SLOW] = slow ? 1u : 0u;
      if (slow) atomicOr(ws.diag, kDiagSlowPath);
    }
  }
  // The streaming pass stored +0 at every candidate (random-k; top-k segments with seg_zc): the
  // exact path needs acc there, which the candidates keep (a row whose candidates did not fit
  // stored acc there itself).  Uniform.
  auto restore_candidates = [&]() {
    if (!e_zero || (KIND == 0 && !T.seg_zc[l])) return;
    for (uint32_t x = a; x < b; ++x) {
      const uint32_t cnt = cc[x];
      const uint32_t sl = T.L == 1 ? first_entry(x, cnt) : ro[x];
      if (sl == kDropped) continue;
      for (uint32_t j = 0; j < cnt; ++j) e_zero[ws.cand_idx[(size_t)sl + j]] = ws.cand_val[(size_t)sl + j];
    }
    __threadfence();
    __syncthreads();
  };
  if (slow) {
    restore_candidates();
    slow_select<KIND>(T, l, data, e_zero, out_idx, out_val, s0, s1, step, hist, lds);
    return;
  }
  const bool rows_lds = nr <= kRowsLds;
  bool tie = false;
  if constexpr (KIND == 0) tie = listed && (R[R_B] == 0 || retry_ties);
  if (tie) {
    // The threshold bin is the key A alone, whose elements the streaming pass counted per row but
    // did not store (a retry: the key A2, counted by k_collect): every stored candidate wins, and
    // the first `need` of the elements equal to it, in index order.  A scan of the rows' tie counts
    // finds the row of the last winner, and one pass over that row's elements in acc the winner
    // itself.  The rows with winning ties are emitted from acc (all their elements are scanned
    // there: counts = the row's length, flagged kAccRow).
    __shared__ uint32_t s_row, s_rank;
    const uint32_t* rt = ws.rtie + r0;
    uint32_t tl[kPer], st = 0;
#pragma unroll
    for (uint32_t x = 0; x < kPer; ++x) {
      tl[x] = a + x < b ? rt[a + x] : 0u;
      st += tl[x];
    }
    for (uint32_t x = a + kPer; x < b; ++x) st += rt[x];
    uint32_t totT;
    uint32_t before = block_excl_scan<kSelNT>(st, lds, totT);
    if (totT < need) {  // a retry with too few ties (the tie bin itself holds at least `need`)
      if (threadIdx.x == 0) {
        R[R_SLOW] = 1u;
        atomicOr(ws.diag, kDiagSlowPath);
      }
      restore_candidates();
      slow_select<KIND>(T, l, data, e_zero, out_idx, out_val, s0, s1, step, hist, lds);
      return;
    }
    uint32_t* rcw = ws.rcnt + r0;
    if (retry_ties) {
      // a retry counted only its certain winners per row: all the row's candidates win here
#pragma unroll
      for (uint32_t x = 0; x < kPer; ++x) cr[x] = cn[x];
      for (uint32_t x = a + kPer; x < b; ++x) rcw[x] = cc[x];
    }
    for (uint32_t x = a; x < b; ++x) {
      uint32_t t = 0;  // tl[x - a] by unrolled selects (a dynamic index would put tl in scratch)
      if (x - a < kPer) {
#pragma unroll
        for (uint32_t y = 0; y < kPer; ++y)
          if (y == x - a) t = tl[y];
      } else {
        t = rt[x];
      }
      const uint32_t take = min(t, need > before ? need - before : 0u);
      if (before < need && need <= before + t) {
        s_row = x;
        s_rank = need - before;
      }
      if (take) {
        uint32_t lo, hi;
        row_bounds(T, r0 + x, lo, hi);
        // the row's own candidate count moves to rtie (the emission finds its candidates with it)
        uint32_t oc = 0;
        if (x - a < kPer) {
#pragma unroll
          for (uint32_t y = 0; y < kPer; ++y)
            if (y == x - a) oc = cn[y];
        } else {
          oc = cc[x];
        }
        ws.rtie[r0 + x] = oc;
        ws.counts[r0 + x] = (hi - lo) | kAccRow;
      }
      if (x - a < kPer) {
        uint32_t now = 0;
#pragma unroll
        for (uint32_t y = 0; y < kPer; ++y)
          if (y == x - a) {
            cr[y] += take;
            now = cr[y];
          }
        // (many-row layouts: k_rowcount keeps the winner count of a row emitted from acc)
        if (take) rcw[x] = now;
      } else {
        rcw[x] += take;  // re-read by this thread below
      }
      before += t;
    }
    __syncthreads();
    uint32_t lo, hi;
    row_bounds(T, r0 + s_row, lo, hi);
    const uint32_t A = retry_ties ? R[R_A2] : R[R_A];
    if (e_zero && T.seg_zc[l] && !R[R_RETRY]) {
      // the pass stored +0 at this row's candidates: back to acc before its elements are searched
      // (+0 has the key of a tie at A = 0)
      const uint32_t row = r0 + s_row, oc = ws.rtie[row];
      const uint32_t co = row_entry(T, ws, row, oc, ws.coff[row]);
      if (co != kDropped)
        for (uint32_t j = threadIdx.x; j < oc; j += kSelNT) e_zero[ws.cand_idx[(size_t)co + j]] = ws.cand_val[(size_t)co + j];
      __threadfence();
      __syncthreads();
    }
    const uint32_t p = block_nth_equal(AccKeys{data + lo}, hi - lo, A, s_rank, lds);
    if (threadIdx.x == 0) {
      R[R_T] = A;
      R[R_IT] = lo + p + 1u;
    }
  }
  if (listed && !tie) {
    const uint32_t o = (uint32_t)T.seg_off[l];
    SubLists lk, li;
    lk.arr = ws.list_key;
    li.arr = ws.list_idx;
    lk.base = li.base = T.seg_lbase[l];
    lk.q = li.q = lq;
    uint32_t m = 0;
#pragma unroll
    for (int c = 0; c < kSubLists; ++c) {
      lk.M[c] = li.M[c] = m;
      m += lc[c];
    }
    lk.M[kSubLists] = li.M[kSubLists] = m;
    if (direct) m = mU;
    const bool in_lds = m <= kListLds;
    // top-k, list staged in LDS: the AND and OR of its keys, taken as they pass through
    uint32_t sand = 0xFFFFFFFFu, sor = 0u;
    if (direct) {
      // round trip 2 (direct lists; every row of the segment is one of kPer per thread): each
      // thread notes the pool entries of its rows' undecided candidates at their list positions,
      // then the pairs are fetched, all loads in flight together
      uint32_t f = exU;
#pragma unroll
      for (uint32_t x = 0; x < kPer; ++x) {
        if (a + x < b)
          for (uint32_t t = 0; t < cn[x] - cr[x]; ++t) s_key[f++] = co[x] + t;
      }
      __syncthreads();
      for (uint32_t f0 = 0; f0 < m; f0 += (uint32_t)kSelNT * 4u) {
        uint2 pr[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint32_t fu = f0 + (uint32_t)u * kSelNT + threadIdx.x;
          pr[u] = make_uint2(0u, 0u);
          if (fu < m) {
            const uint32_t at = s_key[fu];
            pr[u] = ws.pairs[at];
          }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint32_t fu = f0 + (uint32_t)u * kSelNT + threadIdx.x;
          if (fu < m) {
            s_key[fu] = pr[u].x;
            s_idx[fu] = pr[u].y;
          }
        }
      }
    } else if (in_lds) {
      // round trip 2: the listed candidates
      for (uint32_t f0 = 0; f0 < m; f0 += (uint32_t)kSelNT * 4u) {
        uint32_t kx[4], ix[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint32_t f = f0 + (uint32_t)u * kSelNT + threadIdx.x;
          kx[u] = f < m ? lk[f] : 0u;
          ix[u] = f < m ? li[f] : 0u;
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const uint32_t f = f0 + (uint32_t)u * kSelNT + threadIdx.x;
          if (f < m) {
            s_key[f] = kx[u];
            s_idx[f] = ix[u];
            sand &= kx[u];
            sor |= kx[u];
          }
        }
      }
    }
    if (rows_lds)
      for (uint32_t x = threadIdx.x; x < nr; x += kSelNT) s_add[x] = 0;
    __syncthreads();
    // need == 0 (random-k only): the certain winners, keys below ulo, are all the winners
    uint32_t Tk = KIND == 1 ? ~T.seg_ulo[l] : 0u, IT = 0;
    // many-row top-k layouts: ties at the threshold key are ordered by index through the rows
    // (a list of millions of equal keys, as bf16 gradients give, took one workgroup 7-14 ms)
    uint32_t tneed = 0;
    uint32_t* defer = KIND == 0 && BIG ? &tneed : nullptr;
    if (need > 0) {
      if constexpr (KIND == 1) {
        // random-k: every listed key' = ~u has u in [ulo, tau), so its bits above the highest one
        // in which ~(tau - 1) and ~ulo differ are theirs: the prefix the AND / OR sweep over the
        // list finds (1.2 us on ResNet-50 flat) comes from the window itself
        const uint32_t klo = ~(uint32_t)(T.seg_tau[l] - 1u), khi = ~T.seg_ulo[l];
        if (in_lds) list_threshold_ao(s_key, s_idx, m, need, klo, khi, hist, lds, s_g, Tk, IT, defer);
        else list_threshold_ao(lk, li, m, need, klo, khi, hist, lds, s_g, Tk, IT, defer);
      } else if (in_lds) {
        // (the AND / OR taken while staging the list spares a sweep over it: 1.1 us on ResNet-50)
        if (m > kRankList) block_and_or(sand, sor, lds);
        list_threshold_ao(s_key, s_idx, m, need, sand, sor, hist, lds, s_g, Tk, IT, defer);
      } else {
        list_threshold(lk, li, m, need, hist, lds, s_g, Tk, IT, defer);
      }
      // the list's winners join their rows' counts
      const uint32_t c0 = o / kTile;
      for (uint32_t j = threadIdx.x; j < (BIG ? 0u : m); j += kSelNT) {
        const uint32_t k = in_lds ? s_key[j] : lk[j];
        const uint32_t i = in_lds ? s_idx[j] : li[j];
        if (k > Tk || (k == Tk && i < IT)) {
          if (rows_lds) atomicAdd(&s_add[i / kTile - c0], 1u);
          else atomicAdd(&ws.rcnt[r0 + (i / kTile - c0)], 1u);
        }
      }
    }
    if (threadIdx.x == 0) {
      R[R_T] = Tk;
      R[R_IT] = IT;
      if (IT == kTieRows) R[R_NEED] = tneed;
    }
    if (!BIG && !rows_lds) {
      // the additions went to global memory: order them before re-reading the counts
      __threadfence();
      __syncthreads();
#pragma unroll
      for (uint32_t x = 0; x < kPer; ++x) cr[x] = a + x < b ? rc[a + x] : 0u;
    }
    __syncthreads();
  }
  if constexpr (BIG) return;
  // row offsets: exclusive scan of the rows' winner counts (mode 1: every candidate wins)
  const uint32_t* cnt = listed ? rc : cc;
  const bool add = listed && rows_lds && !tie;
  uint32_t w[kPer], sum = 0;
#pragma unroll
  for (uint32_t x = 0; x < kPer; ++x) {
    w[x] = (listed ? cr[x] : cn[x]) + (add && a + x < b ? s_add[a + x] : 0u);
    sum += w[x];
  }
  for (uint32_t x = a + kPer; x < b; ++x) sum += cnt[x] + (add ? s_add[x] : 0u);
  uint32_t tot;
  const uint32_t ex = block_excl_scan<kSelNT>(sum, lds, tot);
  uint32_t run = (uint32_t)T.seg_P[l] + ex;
  uint32_t* roff = ws.roff + r0;
#pragma unroll
  for (uint32_t x = 0; x < kPer; ++x) {
    if (a + x < b) roff[a + x] = run;
    run += w[x];
  }
  for (uint32_t x = a + kPer; x < b; ++x) {
    roff[x] = run;
    run += cnt[x] + (add ? s_add[x] : 0u);
  }
  if (threadIdx.x == 0 && tot != kl) atomicOr(ws.diag, kDiagCount);
}

// Large layouts, per row: how many of the row's candidates win (all of them in mode 1).  One
// wavefront per row, kRowcountU chunks of 64 candidates loaded together, counts by ballots (one
// 256-thread workgroup per row, with a workgroup scan, took 180 us over the 244,141 rows of 1e9
// elements).
constexpr uint32_t kRowcountU = 4;
template <int KIND>
__global__ __launch_bounds__(kNT) void k_rowcount(Tables T, WSel ws0, Batch BT) {
  const WSel ws = ws_at(ws0, (uint64_t)blockIdx.y * BT.ws);
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t row = blockIdx.x * (kNT / 64) + (threadIdx.x >> 6);
  if (row >= (uint32_t)T.nrows) return;
  const int l = T.L == 1 ? 0 : T.row_seg[row];
  const uint32_t* R = res_of(ws, l);
  if (R[R_SLOW]) return;
  const uint32_t cw = ws.counts[row], cnt = cw & ~kAccRow;
  // a row emitted from acc (winning ties): k_select wrote its winner count (its stored candidates,
  // which all win, and the ties it takes)
  if (KIND == 0 && (cw & kAccRow)) return;
  const uint32_t co = row_entry(T, ws, row, cnt, ws.coff[row]);
  uint32_t won = 0, tie = 0;
  bool defer = false;  // ties at T resolved by k_rowscan: count them apart
  if (KIND == 1 || R[R_MODE] == 0) {
    const uint32_t Tk = R[R_T], IT = R[R_IT];
    defer = KIND == 0 && IT == kTieRows;
    const uint32_t* ck = ws.cand_key + co;
    const uint32_t* ci = ws.cand_idx + co;
    for (uint32_t j0 = 0; j0 < cnt; j0 += 64u * kRowcountU) {
      uint32_t k[kRowcountU];
#pragma unroll
      for (uint32_t u = 0; u < kRowcountU; ++u) {
        const uint32_t j = j0 + 64u * u + lane;
        k[u] = j < cnt ? ck[j] : 0u;
      }
#pragma unroll
      for (uint32_t u = 0; u < kRowcountU; ++u) {
        const uint32_t j = j0 + 64u * u + lane;
        const bool in = j < cnt;
        // (the index only for a key equal to the threshold key)
        const bool w = in && (k[u] > Tk || (!defer && k[u] == Tk && ci[j] < IT));
        won += (uint32_t)__popcll(__ballot(w));
        tie += (uint32_t)__popcll(__ballot(in && defer && k[u] == Tk));
      }
    }
  } else {
    won = cnt;
  }
  if (lane == 0) {
    ws.rcnt[row] = won;
    if (defer) ws.rtie[row] = tie;
  }
}

// Large layouts, per segment: message offset of every row (exclusive scan of the winner counts),
// in tiles of kSelNT * 8 rows: coalesced loads into LDS, eight consecutive rows per thread, a
// workgroup scan, coalesced stores.  A top-k segment whose threshold key T is shared by more
// candidates than win (R_IT = kTieRows) first scans the rows' counts of keys equal to T the same
// way: the row where the R_NEED-th falls, then that tie inside the row's candidates (stored in
// index order) give R_IT, and the rows before it add all their ties to their winners, the row
// itself the ties up to that one.
__global__ __launch_bounds__(kSelNT) void k_rowscan(Tables T, WSel ws0, Batch BT) {
  const WSel ws = ws_at(ws0, (uint64_t)blockIdx.y * BT.ws);
  constexpr uint32_t kU = 8, kTl = kSelNT * kU;
  __shared__ uint32_t lds[2 * kSelNT / 64];
  __shared__ uint32_t s_c[kTl + kTl / 32];
  auto pad = [](uint32_t i) { return i + (i >> 5); };
  const int l = blockIdx.x;
  const uint32_t* R = res_of(ws, l);
  if (R[R_SLOW]) return;
  const uint32_t r0 = (uint32_t)T.seg_cbase[l], nr = (uint32_t)T.seg_cbase[l + 1] - r0;
  const uint32_t* cnt = ws.rcnt + r0;
  const uint32_t* rt = ws.rtie + r0;
  uint32_t* roff = ws.roff + r0;
  const bool defer = R[R_IT] == kTieRows;  // uniform
  __shared__ uint32_t s_row, s_rank;
  if (defer) {
    const uint32_t need = R[R_NEED];
    if (threadIdx.x == 0) {
      s_row = nr;
      s_rank = 0;
    }
    uint32_t before = 0;  // ties in earlier tiles
    for (uint32_t t0 = 0; t0 < nr; t0 += kTl) {
      uint32_t v[kU];
#pragma unroll
      for (uint32_t u = 0; u < kU; ++u) {
        const uint32_t x = t0 + u * kSelNT + threadIdx.x;
        v[u] = x < nr ? rt[x] : 0u;
      }
#pragma unroll
      for (uint32_t u = 0; u < kU; ++u) s_c[pad(u * kSelNT + threadIdx.x)] = v[u];
      __syncthreads();
      uint32_t sum = 0;
#pragma unroll
      for (uint32_t u = 0; u < kU; ++u) {
        v[u] = s_c[pad(threadIdx.x * kU + u)];
        sum += v[u];
      }
      uint32_t tot;
      uint32_t run = before + block_excl_scan<kSelNT>(sum, lds, tot);
#pragma unroll
      for (uint32_t u = 0; u < kU; ++u) {
        if (run < need && need <= run + v[u]) {
          s_row = t0 + threadIdx.x * kU + u;
          s_rank = need - run;
        }
        run += v[u];
      }
      before += tot;
      __syncthreads();
    }
    __syncthreads();
    // the s_rank-th key equal to T among the row's candidates (index order): the last winner
    const uint32_t sr = s_row;
    if (sr < nr) {
      const uint32_t row = r0 + sr, c = ws.counts[row];
      const uint32_t co = row_entry(T, ws, row, c, ws.coff[row]);
      const uint32_t p = block_nth_equal(ws.cand_key + co, c, R[R_T], s_rank, lds);
      if (threadIdx.x == 0) res_of(ws, l)[R_IT] = ws.cand_idx[co + p] + 1u;
    }
  }
  uint32_t carry = (uint32_t)T.seg_P[l], total = 0;
  // the offsets pass, with the ties of the rows up to s_row added to their winners or without
  auto offsets = [&](auto with_ties) {
    constexpr bool TI = decltype(with_ties)::value;
    const uint32_t srow = TI ? s_row : 0u, srank = TI ? s_rank : 0u;
    for (uint32_t t0 = 0; t0 < nr; t0 += kTl) {
      uint32_t v[kU];
#pragma unroll
      for (uint32_t u = 0; u < kU; ++u) {
        const uint32_t x = t0 + u * kSelNT + threadIdx.x;
        uint32_t tk = 0;  // ties at T: all of a row before srow win, srank of row srow
        if constexpr (TI) tk = x < srow ? rt[x] : (x == srow ? srank : 0u);
        v[u] = x < nr ? cnt[x] + tk : 0u;
      }
#pragma unroll
      for (uint32_t u = 0; u < kU; ++u) s_c[pad(u * kSelNT + threadIdx.x)] = v[u];
      __syncthreads();
      uint32_t sum = 0;
#pragma unroll
      for (uint32_t u = 0; u < kU; ++u) {
        v[u] = s_c[pad(threadIdx.x * kU + u)];
        sum += v[u];
      }
      uint32_t tot;
      uint32_t run = carry + block_excl_scan<kSelNT>(sum, lds, tot);
#pragma unroll
      for (uint32_t u = 0; u < kU; ++u) {
        s_c[pad(threadIdx.x * kU + u)] = run;
        run += v[u];
      }
      __syncthreads();
#pragma unroll
      for (uint32_t u = 0; u < kU; ++u) {
        const uint32_t x = t0 + u * kSelNT + threadIdx.x;
        if (x < nr) roff[x] = s_c[pad(u * kSelNT + threadIdx.x)];
      }
      __syncthreads();
      carry += tot;
      total += tot;
    }
  };
  if (defer) offsets(std::true_type{});
  else offsets(std::false_type{});
  if (threadIdx.x == 0 && total != (uint32_t)T.seg_k[l]) atomicOr(ws.diag, kDiagCount);
}

// Emission: per row, the winners in index order to the message at the row's offset, and e = +0
// there.  One wavefront per RW consecutive rows: lanes j < RW hold row j's count, offset and
// threshold; the rows' candidates are laid out one after another over the 64 lanes (a wave prefix
// of the counts; each lane finds its row by a binary search over those lanes), so a wavefront
// serves its rows in one or a few passes of 64 candidates, the next pass's loads in flight while
// the current one is written.  A winner's position is its row's offset plus the row's winners
// before it: earlier passes (kept by the row's lane) and a ballot count over the row's lanes in
// this pass.  RW = 16 for random-k (a few candidates per row); for top-k, whose rows in the layers
// of largest magnitude hold hundreds, 1 for one or a few workers and 4 for a batch.  A top-k row
// with winning ties (flagged kAccRow) takes its elements in acc as its candidates.  The step's
// last kernel, it also clears the overflow pool's counters for the next step.
template <uint32_t RW, bool ACC_ROWS>
__global__ __launch_bounds__(kNT) void k_emit(Tables T, WSel ws0, uint32_t* out_idx, float* out_val, Batch BT,
                                              int cand_zeroed) {
  static_assert(RW >= 1 && RW <= 64 && (RW & (RW - 1)) == 0, "one lane per row, a power of two");
  const WSel ws = ws_at(ws0, (uint64_t)blockIdx.y * BT.ws);
  float* e_zero = BT.e[blockIdx.y];
  out_idx = shifted(out_idx, (uint64_t)blockIdx.y * BT.msg * 4u);
  out_val = out_val ? shifted(out_val, (uint64_t)blockIdx.y * BT.msg * 4u) : nullptr;
  const uint32_t lane = threadIdx.x & 63;
  const uint32_t row0 = (blockIdx.x * (kNT / 64) + (threadIdx.x >> 6)) * RW;
  if (row0 >= (uint32_t)T.nrows) return;
  // lane j < RW: row row0 + j (rows past the end and rows of exact-path segments count 0)
  if (blockIdx.x == 0 && threadIdx.x < (unsigned)kPools) *pcnt_of(ws, threadIdx.x) = 0u;
  const uint32_t myrow = row0 + lane;
  const bool has_row = lane < RW && myrow < (uint32_t)T.nrows;
  uint32_t cnt = 0, off = 0, Tk = 0, IT = 0, pend = 0, co = 0, in_acc = 0;
  // rl: the pass stored +0 at this row's candidates (random-k, fused; top-k segments with seg_zc
  // unless a candidate retry put acc back): losers get their values back, winners are left;
  // otherwise winners get +0.  A row emitted from acc whose candidates are +0 first puts them
  // back (rst, ocnt and oco: its own candidates).
  uint32_t rl = 0, rst = 0, ocnt = 0, oco = 0;
  if (has_row) {
    const int l = T.L == 1 ? 0 : T.row_seg[myrow];  // one segment: no load before the record
    const uint32_t* R = res_of(ws, l);
    cnt = ws.counts[myrow];
    co = ws.coff[myrow];
    off = ws.roff[myrow];
    pend = (uint32_t)T.seg_P[l + 1];
    Tk = R[R_T];
    IT = R[R_IT];
    const bool zrow = e_zero && (cand_zeroed || (ACC_ROWS && T.seg_zc[l] && !R[R_RETRY]));
    if (ACC_ROWS && (cnt & kAccRow)) {  // the row's first element in acc
      if (zrow) {
        ocnt = ws.rtie[myrow];
        oco = row_entry(T, ws, myrow, ocnt, co);
        rst = oco != kDropped ? 1u : 0u;
      }
      uint32_t hi;
      row_bounds(T, myrow, co, hi);
      cnt &= ~kAccRow;
      in_acc = 1u;
    } else {
      co = row_entry(T, ws, myrow, cnt, co);
      rl = zrow ? 1u : 0u;
    }
    if (R[R_SLOW]) {
      cnt = 0;
      rst = 0;
    }
  }
  const float* acc = BT.g[blockIdx.y] ? BT.e[blockIdx.y] : BT.src[blockIdx.y];
  if (ACC_ROWS && __ballot(rst != 0u)) {  // wave-uniform
    for (uint32_t u = 0; u < RW; ++u) {
      const uint32_t n = __shfl(rst, (int)u, 64) ? __shfl(ocnt, (int)u, 64) : 0u;
      const uint32_t b0 = __shfl(oco, (int)u, 64);
      for (uint32_t j = lane; j < n; j += 64) e_zero[ws.cand_idx[(size_t)b0 + j]] = ws.cand_val[(size_t)b0 + j];
    }
    __threadfence();  // before the rows' elements are read from acc
  }
  const uint32_t incl = wave_incl_scan(cnt);
  const uint32_t total = __shfl(incl, 63, 64);
  const uint32_t pre = incl - cnt;  // this lane's row: first flattened candidate
  // The wave's loop; the form that tests for rows emitted from acc runs only in a wave holding one.
  auto run = [&](auto acc_rows) {
    constexpr bool AR = decltype(acc_rows)::value;
    // flattened candidate f -> its row lane r (the last row lane with pre_r <= f; for f < total that
    // row's count is nonzero, so f lies inside it) and its entry: a pool entry, or an element of acc
    auto locate = [&](uint32_t f, uint32_t& r, uint32_t& sl, bool& ia) {
      r = 0;
#pragma unroll
      for (uint32_t step = RW / 2; step >= 1; step >>= 1) {
        const uint32_t p = __shfl(pre, (int)(r + step), 64);
        if (f < total && p <= f) r += step;
      }
      sl = __shfl(co, (int)r, 64) + (f - __shfl(pre, (int)r, 64));
      ia = AR && __shfl(in_acc, (int)r, 64) != 0u;
    };
    auto fetch = [&](uint32_t sl, bool ia, uint32_t& k, uint32_t& i, float& v) {
      if (AR && ia) {
        v = acc[sl];
        k = mag_key(v);
        i = sl;
      } else {
        k = ws.cand_key[sl];
        i = ws.cand_idx[sl];
        v = ws.cand_val[sl];
      }
    };
    uint32_t done = 0;  // this lane's row: winners emitted in earlier passes
    uint32_t r, sl;
    bool ia;
    locate(lane, r, sl, ia);
    uint32_t k = 0, i = 0;
    float v = 0.0f;
    if (lane < total) fetch(sl, ia, k, i, v);
    for (uint32_t f0 = 0; f0 < total; f0 += 64) {
      const uint32_t f = f0 + lane;
      const bool in = f < total;
      const uint32_t rpre = __shfl(pre, (int)r, 64);
      const uint32_t rTk = __shfl(Tk, (int)r, 64), rIT = __shfl(IT, (int)r, 64);
      const uint32_t roffr = __shfl(off, (int)r, 64) + __shfl(done, (int)r, 64);
      const uint32_t rpend = __shfl(pend, (int)r, 64), rrl = __shfl(rl, (int)r, 64);
      const uint32_t ck = k, ci = i;
      const float cv = v;
      // the next pass's candidates, in flight while this pass is written
      uint32_t rn = 0, sn = 0;
      bool ian = false;
      locate(f + 64, rn, sn, ian);
      if (f + 64 < total) fetch(sn, ian, k, i, v);
      const bool win = in && (ck > rTk || (ck == rTk && ci < rIT));
      const uint64_t bw = __ballot(win);
      // this pass's lanes of row r before this lane: [lo_r, lane)
      const uint32_t lo_r = rpre > f0 ? rpre - f0 : 0u;
      const uint64_t below = (lane ? (~0ull >> (64 - lane)) : 0ull) & ~((lo_r ? (~0ull >> (64 - lo_r)) : 0ull));
      const uint32_t pos = roffr + (uint32_t)__popcll(bw & below);
      if (win && pos < rpend) {
        out_idx[pos] = ci;
        if (out_val) out_val[pos] = cv;
        if (e_zero && !rrl) e_zero[ci] = 0.0f;
      }
      if (e_zero && rrl && in && !win) e_zero[ci] = cv;  // a losing candidate stored as +0: its value
      // each row lane adds its winners of this pass
      if (has_row) {
        const uint32_t a = pre > f0 ? pre - f0 : 0u, z = incl > f0 ? min(incl - f0, 64u) : 0u;
        if (z > a) {
          const uint64_t m = (z == 64 ? ~0ull : (~0ull >> (64 - z))) & ~(a ? (~0ull >> (64 - a)) : 0ull);
          done += (uint32_t)__popcll(bw & m);
        }
      }
      r = rn;
    }
  };
  if (ACC_ROWS && __ballot(in_acc != 0u)) run(std::true_type{});
  else run(std::false_type{});
}

}  // namespace efs
