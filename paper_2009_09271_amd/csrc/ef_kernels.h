// HIP kernels of the efsparse hot path (gfx950).
//
// Streaming kernels walk the gradient in chunks of kTile elements (one workgroup per chunk,
// kRounds coalesced float4 groups per thread).  A chunk lies in one or more segments; the common
// single-segment case takes uniform fast paths.
//
// Top-k and random-k (Section 3) share one pipeline without any cross-workgroup synchronisation
// inside a kernel:
//   k_topk_sample   top-k only: per segment, a candidate threshold: exact (k-th largest key) for
//                   segments of up to kSampleMax elements, otherwise from a sample of contiguous
//                   runs spread over the segment, set so that the candidates very likely number
//                   at least k_l.
//   k_stream_sel    fused accumulate (acc = g + e, written to e) and candidate test (top-k: key >=
//                   threshold; random-k: Philox key < tau_l, a binomial bound on k_l); every chunk
//                   writes its candidates, in index order, to its own slot plus a count.
//   k_select_emit   one workgroup per segment: gathers the segment's candidates, selects the k_l
//                   winners exactly by radix levels (top-k: largest magnitude key; random-k:
//                   smallest Philox key; ties to the lower index), writes them in index order to
//                   the message and zeroes e there.  A segment with fewer than k_l candidates is
//                   resolved exactly over all of its elements.
// Block-random-k is one fused streaming pass (k_randblock_step).
// The aggregate (Algorithm 1) accumulates each output tile in LDS in worker order.
#pragma once

#include "ef_device.h"

namespace efs {

struct WSel {
  uint32_t* diag;       // [4]   diagnostics bits
  uint32_t* res;        // [L][kResWords]
  uint32_t* counts;     // [nchunks] candidates per chunk
  uint32_t* cofs;       // [2 * ncrows] per segment: compacted non-empty chunk rows (ids, flat offsets)
  uint32_t* cand_idx;   // [nchunks * kTile] per-chunk candidate slots
  float* cand_val;      // [nchunks * kTile]
  uint32_t* cand_key;   // [nchunks * kTile] selection key' of each candidate
  uint32_t* dense_idx;  // [d] candidates of segment l, gathered to [o_l, o_l + N_l)
  float* dense_val;     // [d]
  uint32_t* dense_key;  // [d]
};

__device__ __forceinline__ uint32_t* res_of(const WSel& w, int l) { return w.res + (size_t)l * kResWords; }

// ---------------------------------------------------------------------------------------------
// Utility kernels
// ---------------------------------------------------------------------------------------------
// Algorithm 1 accumulate step: acc = g + e.
template <int GDT>
__global__ __launch_bounds__(kNT) void k_accumulate(int32_t d, const void* g, const float* e, float* acc) {
  const uint32_t lo = blockIdx.x * kTile, hi = min((uint32_t)d, lo + kTile);
  float gv[kRounds][4], ev[kRounds][4];
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    const int nv = i0 < hi ? (int)min(4u, hi - i0) : 0;
    load4g<GDT>(g, i0, nv, gv[r]);
    load4(e, i0, nv, ev[r]);
  }
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    const int nv = i0 < hi ? (int)min(4u, hi - i0) : 0;
    float a[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) a[q] = gv[r][q] + ev[r][q];
    store4(acc, i0, nv, a);
  }
}

__global__ __launch_bounds__(kNT) void k_copy(int32_t d, const float* src, float* dst) {
  const uint32_t lo = blockIdx.x * kTile, hi = min((uint32_t)d, lo + kTile);
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    const int nv = i0 < hi ? (int)min(4u, hi - i0) : 0;
    float v[4];
    load4(src, i0, nv, v);
    store4(dst, i0, nv, v);
  }
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

// Fused worker step: acc = g + e; val[P_l + t] = acc on the run; e' = +0 on the run, acc elsewhere.
template <int GDT>
__global__ __launch_bounds__(kNT) void k_randblock_step(Tables T, const void* g, float* e, uint32_t s0,
                                                        uint32_t s1, uint32_t step, uint32_t* start,
                                                        float* val) {
  const uint32_t c = blockIdx.x;
  const uint32_t lo = c * kTile, hi = min((uint32_t)T.d, lo + kTile);
  const int sf = T.chunk_sf[c], sl = T.chunk_sl[c];
  const bool uni = sf == sl;
  RunSeg rs = run_seg(T, sf, step, s0, s1);
  int cur = sf;
  float gv[kRounds][4], ev[kRounds][4];
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    const int nv = i0 < hi ? (int)min(4u, hi - i0) : 0;
    load4g<GDT>(g, i0, nv, gv[r]);
    load4(e, i0, nv, ev[r]);
  }
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    const int nv = i0 < hi ? (int)min(4u, hi - i0) : 0;
    float out[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float a = gv[r][q] + ev[r][q];
      out[q] = a;
      if (q < nv) {
        const uint32_t i = i0 + q;
        if (!uni) {
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
  }
  // start of every segment that begins in this chunk
  for (int l = sf + (int)threadIdx.x; l <= sl; l += kNT) {
    if ((uint32_t)T.seg_off[l] >= lo)
      start[l] = block_start((uint32_t)l, step, s0, s1, (uint32_t)T.seg_bl[l], (uint32_t)T.seg_nb[l]);
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

// Out-of-place residual update for a block message: e = +0 on the runs, acc elsewhere.
__global__ __launch_bounds__(kNT) void k_block_update(Tables T, const float* acc, const uint32_t* start, float* e) {
  const uint32_t c = blockIdx.x;
  const uint32_t lo = c * kTile, hi = min((uint32_t)T.d, lo + kTile);
  const int sf = T.chunk_sf[c], sl = T.chunk_sl[c];
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    const int nv = i0 < hi ? (int)min(4u, hi - i0) : 0;
    float v[4];
    load4(acc, i0, nv, v);
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
}

// ---------------------------------------------------------------------------------------------
// Aggregate (Algorithm 1): out = (sum over workers in order, from +0) / W.  One workgroup per
// output tile of kTile elements accumulates in LDS; a barrier separates consecutive workers.
// ---------------------------------------------------------------------------------------------
// tile_start[w][tau] = first entry of message w whose index lies in tile >= tau (tau = 0..nt).
// Grid: (ceil(K / kNT), W).
__global__ __launch_bounds__(kNT) void k_agg_ranges(int32_t d, int32_t K, int32_t nt, const uint32_t* idx,
                                                    uint32_t* tile_start) {
  const uint32_t j = blockIdx.x * kNT + threadIdx.x;
  const int w = blockIdx.y;
  if (j >= (uint32_t)K) return;
  const uint32_t* m = idx + (size_t)w * K;
  uint32_t* ts = tile_start + (size_t)w * (nt + 1);
  auto tile = [&](uint32_t i) -> int { return i < (uint32_t)d ? (int)(i / kTile) : nt; };
  const int tj = tile(m[j]);
  const int tp = j == 0 ? -1 : tile(m[j - 1]);
  for (int tau = tp + 1; tau <= tj; ++tau) ts[tau] = j;
  if (j == (uint32_t)K - 1)
    for (int tau = tj + 1; tau <= nt; ++tau) ts[tau] = (uint32_t)K;
}

__device__ __forceinline__ void agg_write(float* out, uint32_t lo, uint32_t hi, const float* acc,
                                          int average, float fW) {
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t x = (uint32_t)(r * kNT + threadIdx.x) * 4u;
    const uint32_t i0 = lo + x;
    const int nv = i0 < hi ? (int)min(4u, hi - i0) : 0;
    float v[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = average ? __fdiv_rn(acc[x + q], fW) : acc[x + q];
    store4(out, i0, nv, v);
  }
}

__global__ __launch_bounds__(kNT) void k_agg_sparse(int32_t d, int32_t W, int32_t K, int32_t nt,
                                                    const uint32_t* idx, const float* val,
                                                    const uint32_t* tile_start, int average, float* out) {
  __shared__ float acc[kTile];
  const uint32_t tau = blockIdx.x;
  const uint32_t lo = tau * kTile, hi = min((uint32_t)d, lo + kTile);
  for (uint32_t x = threadIdx.x; x < kTile; x += kNT) acc[x] = 0.0f;
  __syncthreads();
  for (int w = 0; w < W; ++w) {
    const uint32_t* ts = tile_start + (size_t)w * (nt + 1);
    const uint32_t a = min(ts[tau], (uint32_t)K), b = min(ts[tau + 1], (uint32_t)K);
    const uint32_t* m = idx + (size_t)w * K;
    const float* v = val + (size_t)w * K;
    for (uint32_t j = a + threadIdx.x; j < b; j += kNT) {
      const uint32_t i = m[j];
      if (i >= lo && i < hi) acc[i - lo] += v[j];
    }
    __syncthreads();
  }
  agg_write(out, lo, hi, acc, average, (float)W);
}

__global__ __launch_bounds__(kNT) void k_agg_block(Tables T, int32_t W, int32_t K, const uint32_t* start,
                                                   const float* val, int average, float* out) {
  __shared__ float acc[kTile];
  const uint32_t c = blockIdx.x;
  const uint32_t lo = c * kTile, hi = min((uint32_t)T.d, lo + kTile);
  const int sf = T.chunk_sf[c], sl = T.chunk_sl[c];
  for (uint32_t x = threadIdx.x; x < kTile; x += kNT) acc[x] = 0.0f;
  __syncthreads();
  for (int w = 0; w < W; ++w) {
    const uint32_t* st = start + (size_t)w * T.L;
    const float* v = val + (size_t)w * K;
    for (int l = sf; l <= sl; ++l) {
      const uint32_t o = T.seg_off[l], n = T.seg_off[l + 1] - o, k = T.seg_k[l], P = T.seg_P[l];
      const uint32_t s = st[l] % n;
      // run piece 1: local [s, min(s + k, n)), t = j - s;  piece 2: local [0, s + k - n), t = j + n - s
      const uint32_t e1 = min(s + k, n);
      const uint32_t a1 = max(lo, o + s), b1 = min(hi, o + e1);
      for (uint32_t i = a1 + threadIdx.x; i < b1; i += kNT) acc[i - lo] += v[P + (i - o - s)];
      if (s + k > n) {
        const uint32_t a2 = max(lo, o), b2 = min(hi, o + (s + k - n));
        for (uint32_t i = a2 + threadIdx.x; i < b2; i += kNT) acc[i - lo] += v[P + (i - o + n - s)];
      }
    }
    __syncthreads();
  }
  agg_write(out, lo, hi, acc, average, (float)W);
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
constexpr uint32_t kKeysLds = 28672;   // candidate keys held in LDS (larger sets stay in global memory)
constexpr uint32_t kCofsLds = 4096;    // chunk rows whose flat offsets stay in LDS

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

// Calls fn(key) for every keys[f], f < n, in a strided order with kBatch loads in flight.
template <typename F>
__device__ __forceinline__ void for_keys(const uint32_t* keys, uint32_t n, F fn) {
  for (uint32_t base = 0; base < n; base += (uint32_t)kSelNT * kBatch) {
    uint32_t k[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const uint32_t f = base + (uint32_t)u * kSelNT + threadIdx.x;
      k[u] = f < n ? keys[f] : 0u;
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const uint32_t f = base + (uint32_t)u * kSelNT + threadIdx.x;
      if (f < n) fn(k[u]);
    }
  }
}

// Radix selection of the need-th largest of n keys: returns T and r such that the winners are
// the keys > T plus the first r keys == T.  kand / kor are the AND and OR of all keys; the levels
// (11 bits each) start at the highest bit in which the keys differ, so concentrated keys still
// spread over the histogram.
__device__ void block_select(const uint32_t* keys, uint32_t n, uint32_t need, uint32_t kand, uint32_t kor,
                             uint32_t* hist, uint32_t* lds, uint32_t& T_out, uint32_t& r_out) {
  const uint32_t diff = kand ^ kor;
  if (diff == 0) {  // all keys equal
    T_out = kand;
    r_out = need;
    return;
  }
  const int h = 31 - __clz(diff);
  uint32_t prefix = h == 31 ? 0u : (kand & (0xFFFFFFFFu << (h + 1)));
  int known = 31 - h;
  while (known < 32) {
    const int w = min(11, 32 - known);
    const int shift = 32 - known - w;
    for (int b = threadIdx.x; b < (1 << w); b += kSelNT) hist[b] = 0;
    __syncthreads();
    const uint32_t pmask = known == 0 ? 0u : (0xFFFFFFFFu << (32 - known));
    const uint32_t want = prefix & pmask;
    for_keys(keys, n, [&](uint32_t k) {
      if ((k & pmask) == want) atomicAdd(&hist[(k >> shift) & ((1u << w) - 1u)], 1u);
    });
    __syncthreads();
    uint32_t above;
    const int bin = block_resolve<kSelNT>(hist, 1 << w, need, lds, above);
    prefix |= (uint32_t)max(bin, 0) << shift;
    need -= above;
    known += w;
  }
  T_out = prefix;
  r_out = need;
}

// Top-k candidate threshold per segment (one workgroup per segment): the lower edge of the
// 11-bit histogram bin (starting at the highest bit in which the sampled keys differ) that holds
// the rank-th largest sampled key.  Exact k-th largest key when the whole segment fits the sample.
template <int GDT, bool FUSED>
__global__ __launch_bounds__(kSelNT) void k_topk_sample(Tables T, const void* g, const float* src, WSel ws) {
  constexpr uint32_t runs = kSampleMax / kSampleRun;
  __shared__ uint32_t keys[kSampleMax];
  __shared__ uint32_t hist[kHBins];
  __shared__ uint32_t lds[2 * kSelNT / 64];
  __shared__ uint32_t run_start[runs];
  const int l = blockIdx.x;
  const uint32_t o = (uint32_t)T.seg_off[l], n = (uint32_t)T.seg_off[l + 1] - o;
  EFS_PHASE(8);
  constexpr int per = kSampleMax / kSelNT;
  const bool exact = n <= (uint32_t)kSampleMax;
  const uint32_t m = exact ? n : (uint32_t)kSampleMax;
  const uint32_t rank = exact ? (uint32_t)T.seg_k[l] : (uint32_t)T.seg_srank[l];
  // runs of kSampleRun contiguous elements, evenly spaced over the segment
  if (!exact && threadIdx.x < runs)
    run_start[threadIdx.x] = o + (uint32_t)(((uint64_t)threadIdx.x * (n - kSampleRun)) / (runs - 1));
  __syncthreads();
  float a[per];
#pragma unroll
  for (int u = 0; u < per; ++u) {
    const uint32_t j = (uint32_t)(u * kSelNT) + threadIdx.x;
    const uint32_t i = exact ? o + j : run_start[j / kSampleRun] + j % kSampleRun;
    a[u] = 0.0f;
    if (j < m) {
      if constexpr (FUSED) a[u] = load1g<GDT>(g, i) + src[i];
      else a[u] = src[i];
    }
  }
  uint32_t kand = 0xFFFFFFFFu, kor = 0u;
#pragma unroll
  for (int u = 0; u < per; ++u) {
    const uint32_t j = (uint32_t)(u * kSelNT) + threadIdx.x;
    if (j < m) {
      const uint32_t k = mag_key(a[u]);
      keys[j] = k;
      kand &= k;
      kor |= k;
    }
  }
  block_and_or(kand, kor, lds);
  EFS_PHASE(9);
  uint32_t thr;
  if (exact) {
    uint32_t r_unused;
    block_select(keys, m, rank, kand, kor, hist, lds, thr, r_unused);
  } else if (kand == kor) {
    thr = kand;
  } else {
    const int h = 31 - __clz(kand ^ kor);
    const int w = min(11, h + 1), shift = h + 1 - w;
    const uint32_t prefix = h == 31 ? 0u : (kand & (0xFFFFFFFFu << (h + 1)));
    for (int b = threadIdx.x; b < (1 << w); b += kSelNT) hist[b] = 0;
    __syncthreads();
    for_keys(keys, m, [&](uint32_t k) { atomicAdd(&hist[(k >> shift) & ((1u << w) - 1u)], 1u); });
    __syncthreads();
    uint32_t above;
    const int bin = block_resolve<kSelNT>(hist, 1 << w, rank, lds, above);
    thr = prefix | ((uint32_t)max(bin, 0) << shift);
  }
  EFS_PHASE(11);
  if (threadIdx.x == 0) res_of(ws, l)[R_THR] = thr;
}

// Fused accumulate + candidate test + per-chunk ordered compaction into the chunk's slot.
template <int KIND, int GDT, bool FUSED>
__global__ __launch_bounds__(kNT) void k_stream_sel(Tables T, const void* g, const float* src, float* acc_out,
                                                    uint32_t s0, uint32_t s1, uint32_t step, WSel ws) {
  __shared__ uint32_t wt[kRounds][kNT / 64];
  const uint32_t c = blockIdx.x;
  const uint32_t lo = c * kTile, hi = min((uint32_t)T.d, lo + kTile);
  const int sf = T.chunk_sf[c], sl = T.chunk_sl[c];
  const bool uni = sf == sl;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const uint32_t o_u = (uint32_t)T.seg_off[sf];
  uint32_t thr_u = 0;
  uint64_t tau_u = 0;
  if constexpr (KIND == 0) thr_u = res_of(ws, sf)[R_THR];
  else tau_u = T.seg_tau[sf];
  const bool aligned = uni && (o_u & 3u) == 0;

  float v[kRounds][4];
  if constexpr (FUSED) {
    float gv[kRounds][4];
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
      const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
      const int nv = i0 < hi ? (int)min(4u, hi - i0) : 0;
      load4g<GDT>(g, i0, nv, gv[r]);
      load4(src, i0, nv, v[r]);
    }
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
      const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
      const int nv = i0 < hi ? (int)min(4u, hi - i0) : 0;
#pragma unroll
      for (int q = 0; q < 4; ++q) v[r][q] = gv[r][q] + v[r][q];
      store4(acc_out, i0, nv, v[r]);
    }
  } else {
#pragma unroll
    for (int r = 0; r < kRounds; ++r) {
      const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
      const int nv = i0 < hi ? (int)min(4u, hi - i0) : 0;
      load4(src, i0, nv, v[r]);
    }
  }
  // candidate flags; wave-level prefixes through ballots, one barrier for the whole chunk
  uint32_t mask[kRounds], lpre[kRounds];
  uint32_t kk[kRounds][4];  // key' of each element (random-k: ~Philox key)
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    const int nv = i0 < hi ? (int)min(4u, hi - i0) : 0;
    uint32_t mk = 0;
    if constexpr (KIND == 0) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        kk[r][q] = mag_key(v[r][q]);
        if (q < nv) {
          uint32_t thr = thr_u;
          if (!uni) thr = res_of(ws, seg_of(i0 + q, sf, sl, T.seg_off))[R_THR];
          if (kk[r][q] >= thr) mk |= 1u << q;
        }
      }
    } else {
      if (aligned) {
        uint4 x = make_uint4(0u, 0u, 0u, 0u);
        if (nv > 0) x = philox(make_uint4((i0 - o_u) >> 2, 0u, step, kRandkTag | (uint32_t)sf), s0, s1);
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          kk[r][q] = ~word(x, q);
          if (q < nv && (uint64_t)word(x, q) < tau_u) mk |= 1u << q;
        }
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          kk[r][q] = 0u;
          if (q < nv) {
            const uint32_t i = i0 + q;
            const int l = uni ? sf : seg_of(i, sf, sl, T.seg_off);
            const uint32_t u = randk_key(i - (uint32_t)T.seg_off[l], (uint32_t)l, step, s0, s1);
            kk[r][q] = ~u;
            if ((uint64_t)u < T.seg_tau[l]) mk |= 1u << q;
          }
        }
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
  }
  __syncthreads();
  uint32_t base = 0;
  uint32_t* cidx = ws.cand_idx + (size_t)c * kTile;
  float* cval = ws.cand_val + (size_t)c * kTile;
  uint32_t* ckey = ws.cand_key + (size_t)c * kTile;
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    uint32_t rb = base;
#pragma unroll
    for (int w = 0; w < kNT / 64; ++w) rb += w < wid ? wt[r][w] : 0u;
    if (mask[r]) {
      const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
      uint32_t pos = rb + lpre[r];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        if ((mask[r] >> q) & 1u) {
          cidx[pos] = i0 + q;
          cval[pos] = v[r][q];
          ckey[pos] = kk[r][q];
          ++pos;
        }
      }
    }
#pragma unroll
    for (int w = 0; w < kNT / 64; ++w) base += wt[r][w];
  }
  if (threadIdx.x == 0) ws.counts[c] = base;
}

// Exact selection over the whole segment (used when the candidates cannot contain the answer):
// radix levels over the keys of all d_l elements, then an index-ordered emission.
template <int KIND>
__device__ void slow_select(const Tables& T, int l, const float* data, float* e_zero, uint32_t* out_idx,
                            float* out_val, uint32_t s0, uint32_t s1, uint32_t step, uint32_t* hist, uint32_t* lds) {
  const uint32_t o = (uint32_t)T.seg_off[l], n = (uint32_t)T.seg_off[l + 1] - o;
  const uint32_t P = (uint32_t)T.seg_P[l], kl = (uint32_t)T.seg_k[l];
  auto keyat = [&](uint32_t j) -> uint32_t { return sel_key<KIND>(o + j, data[o + j], o, l, step, s0, s1); };
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
      out_val[pos] = data[o + j];
      if (e_zero) e_zero[o + j] = 0.0f;
    }
    run_a += tot & 0xFFFFu;
    run_b += tot >> 16;
  }
}

// Per-segment exact selection among the candidates in the chunk slots, and the emission of the
// k_l winners in index order (one workgroup per segment).  Every pass is wave-contiguous: wave w
// owns a contiguous share of the flat (= index) order of the candidates and walks it 64 entries at
// a time with kBatch loads in flight, so accesses stay coalesced.  The gather copies the
// candidates to dense arrays at [o_l, o_l + N) (N <= d_l; keys to LDS when they fit), the radix
// levels sweep the keys, and the emission uses in-wave ballot prefixes plus one scan of the wave
// totals.  The row offsets and keys live either in LDS or in global memory; each placement is its
// own instantiation so that every access has a known address space (no flat accesses, whose waits
// would serialise the batches).
// Last position m >= i with off[m] <= f (off strictly increasing over [0, n); off[i] <= f).
__device__ __forceinline__ uint32_t advance_row(const uint32_t* off, uint32_t n, uint32_t i, uint32_t f) {
  if (i + 1 >= n || off[i + 1] > f) return i;
  uint32_t lo = i + 1, hi, step = 1;
  while (true) {  // gallop until off[hi] > f
    hi = lo + step;
    if (hi >= n) {
      hi = n;
      break;
    }
    if (off[hi] > f) break;
    lo = hi;
    step <<= 1;
  }
  while (hi - lo > 1) {
    const uint32_t mid = (lo + hi) >> 1;
    if (off[mid] <= f) lo = mid; else hi = mid;
  }
  return lo;
}

struct SelSeg {
  int l;
  uint32_t o, kl, P, c0, nc, a0, b1, N;
};

template <int KIND, bool KEYS_LDS>
__device__ __forceinline__ void select_emit_tail(const Tables& T, const WSel& ws, const SelSeg& S, const uint32_t* crow,
                                                 const uint32_t* coff, uint32_t nnz, uint32_t* keys, float* e_zero,
                                                 uint32_t* out_idx, float* out_val, uint32_t* hist, uint32_t* lds,
                                                 uint32_t (*s_wtot)[kSelNT / 64]) {
  constexpr int NW = kSelNT / 64;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const uint32_t N = S.N;
  const uint32_t W0 = (uint32_t)(((uint64_t)N * wid) / NW), W1 = (uint32_t)(((uint64_t)N * (wid + 1)) / NW);
  uint32_t* didx = ws.dense_idx + S.o;
  float* dval = ws.dense_val + S.o;
  // gather
  uint32_t kand = 0xFFFFFFFFu, kor = 0u;
  {
    // m0: the non-empty row holding the wave's next flat position (wave-uniform).  For 64
    // consecutive positions the rows involved are m0 .. m0+63 at most (every row is non-empty):
    // each lane loads one row boundary and finds its own row by a shuffle binary search.
    uint32_t m0 = advance_row(coff, nnz, 0, W0 < W1 ? W0 : 0u);
    for (uint32_t base = W0; base < W1; base += 64u * kBatch) {
      size_t at[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const uint32_t fb = base + (uint32_t)u * 64u;  // wave-uniform
        const uint32_t f = fb + lane;
        const uint32_t mb = m0 + lane;
        const uint32_t bnd = mb < nnz ? coff[mb] : 0xFFFFFFFFu;
        const uint32_t rid = mb < nnz ? crow[mb] : 0u;
        uint32_t j = 0;  // last j with boundary(m0 + j) <= f
#pragma unroll
        for (int st = 32; st > 0; st >>= 1) {
          const uint32_t cand = j + (uint32_t)st;
          const uint32_t bc = __shfl(bnd, (int)min(cand, 63u), 64);
          if (cand < 64u && bc <= f) j = cand;
        }
        const uint32_t row = __shfl(rid, (int)j, 64), off = __shfl(bnd, (int)j, 64);
        at[u] = f < W1 ? (size_t)(S.c0 + row) * kTile + (row == 0 ? S.a0 : 0u) + (f - off) : 0;
        // row of the next wave-step's first position (fb + 64): lane 63's row, or the one after
        const uint32_t j63 = __shfl(j, 63, 64);
        uint32_t nb = __shfl(bnd, (int)min(j63 + 1u, 63u), 64);
        if (j63 == 63u) nb = m0 + 64u < nnz ? coff[m0 + 64u] : 0xFFFFFFFFu;  // every row held one position
        m0 += j63 + (nb <= fb + 64u ? 1u : 0u);
      }
      uint32_t ci[kBatch], ck[kBatch];
      float cv[kBatch];
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const bool in = base + (uint32_t)u * 64u + lane < W1;
        ci[u] = in ? ws.cand_idx[at[u]] : 0u;
        cv[u] = in ? ws.cand_val[at[u]] : 0.0f;
        ck[u] = in ? ws.cand_key[at[u]] : 0u;
      }
#pragma unroll
      for (int u = 0; u < kBatch; ++u) {
        const uint32_t f = base + (uint32_t)u * 64u + lane;
        if (f < W1) {
          didx[f] = ci[u];
          dval[f] = cv[u];
          keys[f] = ck[u];
          kand &= ck[u];
          kor |= ck[u];
        }
      }
    }
  }
  block_and_or(kand, kor, lds);  // also makes the gathered data visible to the workgroup
  EFS_PHASE(3);
  uint32_t Tk, r;
  block_select(keys, N, S.kl, kand, kor, hist, lds, Tk, r);
  EFS_PHASE(4);
  // emission in flat (= index) order
  uint32_t na = 0, nb = 0;
  for (uint32_t base = W0; base < W1; base += 64u * kBatch) {
    uint32_t k[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const uint32_t f = base + (uint32_t)u * 64u + lane;
      k[u] = f < W1 ? keys[f] : 0u;
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const bool in = base + (uint32_t)u * 64u + lane < W1;
      na += (uint32_t)__popcll(__ballot(in && k[u] > Tk));
      nb += (uint32_t)__popcll(__ballot(in && k[u] == Tk));
    }
  }
  if (lane == 0) {
    s_wtot[0][wid] = na;
    s_wtot[1][wid] = nb;
  }
  __syncthreads();
  uint32_t ra = 0, rb = 0;
  for (int w = 0; w < wid; ++w) {
    ra += s_wtot[0][w];
    rb += s_wtot[1][w];
  }
  EFS_PHASE(5);
  for (uint32_t base = W0; base < W1; base += 64u * kBatch) {
    uint32_t k[kBatch], ix[kBatch];
    float vv[kBatch];
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const uint32_t f = base + (uint32_t)u * 64u + lane;
      const bool in = f < W1;
      k[u] = in ? keys[f] : 0u;
      ix[u] = in ? didx[f] : 0u;
      vv[u] = in ? dval[f] : 0.0f;
    }
#pragma unroll
    for (int u = 0; u < kBatch; ++u) {
      const bool in = base + (uint32_t)u * 64u + lane < W1;
      const bool a = in && k[u] > Tk, b = in && k[u] == Tk;
      const uint64_t ma = __ballot(a), mb = __ballot(b);
      const uint32_t ea = ra + lanes_below(ma), eb = rb + lanes_below(mb);
      if ((a || (b && eb < r)) && ea + min(eb, r) < S.kl) {
        const uint32_t pos = S.P + ea + min(eb, r);
        out_idx[pos] = ix[u];
        out_val[pos] = vv[u];
        if (e_zero && ix[u] < (uint32_t)T.d) e_zero[ix[u]] = 0.0f;
      }
      ra += (uint32_t)__popcll(ma);
      rb += (uint32_t)__popcll(mb);
    }
  }
  EFS_PHASE(6);
  if (threadIdx.x == 0) {
    uint32_t* R = res_of(ws, S.l);
    R[R_T] = Tk;
    R[R_R] = r;
    R[R_N] = N;
    R[R_SLOW] = 0;
  }
}

// Row offsets of the segment's candidates, then either the exact whole-segment path (too few
// candidates) or the selection over the candidates.
template <int KIND, bool COFS_LDS>
__device__ __forceinline__ void select_emit_body(const Tables& T, const WSel& ws, SelSeg S, uint32_t* crow,
                                                 uint32_t* coff, const float* data, float* e_zero, uint32_t* out_idx,
                                                 float* out_val, uint32_t s0, uint32_t s1, uint32_t step,
                                                 uint32_t* hist, uint32_t* lds, uint32_t* s_keys,
                                                 uint32_t (*s_wtot)[kSelNT / 64]) {
  // non-empty chunk rows of the segment, compacted: crow = row id, coff = flat offset of its first
  // candidate (strictly increasing)
  uint32_t N = 0, nnz = 0;
  for (uint32_t i0 = 0; i0 < S.nc; i0 += kSelNT) {
    const uint32_t i = i0 + threadIdx.x;
    uint32_t cnt = 0;
    if (i < S.nc) cnt = (i == S.nc - 1 ? S.b1 : ws.counts[S.c0 + i]) - (i == 0 ? S.a0 : 0u);
    uint32_t tot, totn;
    const uint32_t ex = block_excl_scan<kSelNT>(cnt, lds, tot);
    const uint32_t exn = block_excl_scan<kSelNT>(cnt ? 1u : 0u, lds, totn);
    if (cnt) {
      crow[nnz + exn] = i;
      coff[nnz + exn] = N + ex;
    }
    N += tot;
    nnz += totn;
  }
  S.N = N;
  if (N < S.kl) {  // the candidates cannot hold the answer: exact pass over the whole segment
    slow_select<KIND>(T, S.l, data, e_zero, out_idx, out_val, s0, s1, step, hist, lds);
    if (threadIdx.x == 0) {
      uint32_t* R = res_of(ws, S.l);
      R[R_SLOW] = 1;
      R[R_N] = N;
      atomicOr(ws.diag, kDiagSlowPath);
    }
    return;
  }
  __syncthreads();
  EFS_PHASE(2);
  if (N <= kKeysLds)
    select_emit_tail<KIND, true>(T, ws, S, crow, coff, nnz, s_keys, e_zero, out_idx, out_val, hist, lds, s_wtot);
  else
    select_emit_tail<KIND, false>(T, ws, S, crow, coff, nnz, ws.dense_key + S.o, e_zero, out_idx, out_val, hist, lds,
                                  s_wtot);
}

template <int KIND>
__global__ __launch_bounds__(kSelNT) void k_select_emit(Tables T, WSel ws, const float* data, float* e_zero,
                                                        uint32_t* out_idx, float* out_val, uint32_t s0,
                                                        uint32_t s1, uint32_t step) {
  constexpr int NW = kSelNT / 64;
  __shared__ uint32_t hist[kHBins];
  __shared__ uint32_t lds[2 * NW];
  __shared__ uint32_t s_crow[kCofsLds];
  __shared__ uint32_t s_coff[kCofsLds];
  __shared__ uint32_t s_keys[kKeysLds];
  __shared__ uint32_t s_wtot[2][NW];
  __shared__ uint32_t s_a0, s_b1;
  SelSeg S;
  S.l = blockIdx.x;
  S.o = (uint32_t)T.seg_off[S.l];
  const uint32_t e_ = (uint32_t)T.seg_off[S.l + 1];
  S.kl = (uint32_t)T.seg_k[S.l];
  S.P = (uint32_t)T.seg_P[S.l];
  S.c0 = S.o / kTile;
  S.nc = (e_ - 1) / kTile - S.c0 + 1;
  const uint32_t c1 = S.c0 + S.nc - 1;
  EFS_PHASE(0);
  // candidates of this segment inside its first and last chunk (other segments may share them)
  if (threadIdx.x == 0)
    s_a0 = S.o > S.c0 * kTile ? lower_bound_u32(ws.cand_idx + (size_t)S.c0 * kTile, ws.counts[S.c0], S.o) : 0u;
  if (threadIdx.x == 1)
    s_b1 = e_ < min((uint32_t)T.d, (c1 + 1) * kTile)
               ? lower_bound_u32(ws.cand_idx + (size_t)c1 * kTile, ws.counts[c1], e_)
               : ws.counts[c1];
  __syncthreads();
  S.a0 = s_a0;
  S.b1 = s_b1;
  S.N = 0;
  EFS_PHASE(1);
  if (S.nc <= kCofsLds)
    select_emit_body<KIND, true>(T, ws, S, s_crow, s_coff, data, e_zero, out_idx, out_val, s0, s1, step, hist, lds,
                                 s_keys, s_wtot);
  else
    select_emit_body<KIND, false>(T, ws, S, ws.cofs + 2 * (size_t)T.seg_cbase[S.l], ws.cofs + 2 * (size_t)T.seg_cbase[S.l] + S.nc,
                                  data, e_zero, out_idx, out_val, s0, s1, step, hist, lds, s_keys, s_wtot);
}

}  // namespace efs
