// HIP kernels of the efsparse hot path (gfx950).
//
// Streaming kernels walk the gradient in chunks of kTile elements (one workgroup per chunk,
// kRounds float4 groups per thread, coalesced).  A chunk lies in one or more segments; the
// common single-segment case takes uniform fast paths.
//
// Top-k (Section 3) is an exact radix selection on the 31-bit magnitude key:
//   level 0  (bits 30:20) histogram fused into the accumulate pass      k_topk_hist
//   level 1  (bits 19:10) over the candidate list, emitted in index
//            order with a decoupled look-back                            k_topk_emit
//   level 2  (bits 9:0)   over the list                                 k_list_level
//   emission of the k_l winners in index order                           k_list_emit
// Random-k (Section 3) draws Philox keys in the accumulate pass, keeps keys below a per-segment
// bound as candidates (k_randk_stream), then resolves the exact k_l smallest keys on the list
// (k_list_level) and emits them (k_list_emit).  A segment whose list cannot hold the answer is
// resolved by an exact single-workgroup path over the whole segment.
// Block-random-k (Section 3) is one fused streaming pass (k_randblock_step).
// The aggregate (Algorithm 1) accumulates each output tile in LDS in worker order.
#pragma once

#include "ef_device.h"

namespace efs {

struct WS {
  uint32_t* diag;      // [1] diagnostics bits
  uint32_t* tickets;   // [3] chunk tickets (stream / emit)
  uint32_t* arrive;    // [3][L] per-level arrival counters
  uint32_t* res;       // [L][kResWords]
  uint32_t* cnt;       // [L] random-k candidate counts
  uint32_t* hist;      // [3][L][kHBins]
  uint64_t* st_stream; // [nchunks] look-back words of the streaming pass
  uint64_t* st_emit;   // [n list chunks] look-back words of the emission
  uint32_t* list_idx;  // [cap]
  float* list_val;     // [cap]
  uint32_t* list_key;  // [cap] random-k keys
};

__device__ __forceinline__ uint32_t* hist_row(const WS& w, int slot, int L, int l) {
  return w.hist + ((size_t)slot * L + l) * kHBins;
}
__device__ __forceinline__ uint32_t* res_of(const WS& w, int l) { return w.res + (size_t)l * kResWords; }

// ---------------------------------------------------------------------------------------------
// Utility kernels
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kNT) void k_fill_zero(uint32_t* p, size_t nwords) {
  const size_t n4 = nwords >> 2;
  const size_t stride = (size_t)gridDim.x * kNT;
  for (size_t i = (size_t)blockIdx.x * kNT + threadIdx.x; i < n4; i += stride)
    reinterpret_cast<uint4*>(p)[i] = make_uint4(0, 0, 0, 0);
  for (size_t i = (n4 << 2) + (size_t)blockIdx.x * kNT + threadIdx.x; i < nwords; i += stride) p[i] = 0;
}

// Algorithm 1 accumulate step: acc = g + e.
template <int GDT>
__global__ __launch_bounds__(kNT) void k_accumulate(int32_t d, const void* g, const float* e, float* acc) {
  const uint32_t lo = blockIdx.x * kTile, hi = min((uint32_t)d, lo + kTile);
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    if (i0 >= hi) break;
    const int nv = (int)min(4u, hi - i0);
    float gv[4], ev[4], a[4];
    load4g<GDT>(g, i0, nv, gv);
    load4(e, i0, nv, ev);
#pragma unroll
    for (int q = 0; q < 4; ++q) a[q] = gv[q] + ev[q];
    store4(acc, i0, nv, a);
  }
}

__global__ __launch_bounds__(kNT) void k_copy(int32_t d, const float* src, float* dst) {
  const uint32_t lo = blockIdx.x * kTile, hi = min((uint32_t)d, lo + kTile);
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    if (i0 >= hi) break;
    const int nv = (int)min(4u, hi - i0);
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
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    if (i0 >= hi) break;
    const int nv = (int)min(4u, hi - i0);
    float gv[4], ev[4], out[4];
    load4g<GDT>(g, i0, nv, gv);
    load4(e, i0, nv, ev);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float a = gv[q] + ev[q];
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
    if (i0 >= hi) break;
    const int nv = (int)min(4u, hi - i0);
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
__global__ __launch_bounds__(kNT) void k_agg_ranges(int32_t d, int32_t W, int32_t K, int32_t nt,
                                                    const uint32_t* idx, uint32_t* tile_start) {
  const size_t gid = (size_t)blockIdx.x * kNT + threadIdx.x;
  if (gid >= (size_t)W * K) return;
  const int w = (int)(gid / (uint32_t)K), j = (int)(gid % (uint32_t)K);
  const uint32_t* m = idx + (size_t)w * K;
  uint32_t* ts = tile_start + (size_t)w * (nt + 1);
  auto tile = [&](uint32_t i) -> int { return i < (uint32_t)d ? (int)(i / kTile) : nt; };
  const int tj = tile(m[j]);
  const int tp = j == 0 ? -1 : tile(m[j - 1]);
  for (int tau = tp + 1; tau <= tj; ++tau) ts[tau] = (uint32_t)j;
  if (j == K - 1)
    for (int tau = tj + 1; tau <= nt; ++tau) ts[tau] = (uint32_t)K;
}

__device__ __forceinline__ void agg_write(float* out, uint32_t lo, uint32_t hi, const float* acc,
                                          int average, float fW) {
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t x = (uint32_t)(r * kNT + threadIdx.x) * 4u;
    const uint32_t i0 = lo + x;
    if (i0 >= hi) break;
    const int nv = (int)min(4u, hi - i0);
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
// Shared pieces of the selection kernels
// ---------------------------------------------------------------------------------------------
// Arrival at the end of a pass: every chunk counts itself in for each segment it touched; the
// chunk that completes a segment's count runs `fn(l)` (block-wide) for it.
template <typename F>
__device__ void arrive_and_resolve(uint32_t* arrive, const int32_t* total, int sf, int sl, F fn) {
  __shared__ uint32_t last[kNT];
  __threadfence();
  __syncthreads();
  for (int base = sf; base <= sl; base += kNT) {
    const int l = base + (int)threadIdx.x;
    uint32_t is_last = 0;
    if (l <= sl) is_last = atomicAdd(arrive + l, 1u) == (uint32_t)total[l] - 1u;
    last[threadIdx.x] = is_last;
    __syncthreads();
    const int n = min(kNT, sl - base + 1);
    for (int t = 0; t < n; ++t) {
      if (last[t]) {
        __threadfence();
        fn(base + t);
      }
    }
    __syncthreads();
  }
}

// Exclusive prefix (within the chunk) of flags at element position x, from the per-group table
// gp[g] = (prefix of the group << 4) | (flag bits of its 4 elements).
__device__ __forceinline__ uint32_t chunk_prefix(const uint32_t* gp, uint32_t x, uint32_t ngroups, uint32_t total) {
  const uint32_t g = x >> 2;
  if (g >= ngroups) return total;
  const uint32_t v = gp[g];
  return (v >> 4) + __popc(v & ((1u << (x & 3)) - 1u));
}

// Shared tail of the candidate-emitting streaming passes (top-k level-1 list, random-k
// candidates): given per-element flags for the thread's kRounds groups, computes index-ordered
// list positions per segment (prefix within the chunk + look-back across chunks).
struct EmitCtx {
  uint32_t c, lo, hi;
  int sf, sl;
  uint32_t excl_sf;   // count of the segment sf's flagged elements in earlier chunks
};

__device__ void ordered_positions(const Tables& T, uint64_t* status, uint32_t* diag, EmitCtx& E,
                                  const uint32_t (&mask)[kRounds], uint32_t (&gpre)[kRounds],
                                  uint32_t* gp, uint32_t* lds, uint32_t& total_out) {
  __shared__ uint32_t s_excl;
  uint32_t base = 0;
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    uint32_t tot;
    const uint32_t ex = block_excl_scan((uint32_t)__popc(mask[r]), lds, tot);
    gpre[r] = base + ex;
    gp[r * kNT + threadIdx.x] = ((base + ex) << 4) | mask[r];
    base += tot;
  }
  __syncthreads();
  const uint32_t total = base;
  total_out = total;
  const uint32_t ngroups = kTile / 4;
  const uint32_t o_sl = (uint32_t)T.seg_off[E.sl];
  const uint32_t start_sl = max(o_sl, E.lo);
  const uint32_t cnt_sl = total - chunk_prefix(gp, start_sl - E.lo, ngroups, total);
  const bool sl_cont = o_sl < E.lo;             // segment sl began in an earlier chunk (so sf == sl)
  const uint32_t o_sf = (uint32_t)T.seg_off[E.sf];
  const bool need_lb = o_sf < E.lo;
  if (threadIdx.x == 0) {
    lb_publish(status + E.c, sl_cont ? 1u : 2u, cnt_sl, 0u);
    s_excl = 0;
  }
  if (need_lb && threadIdx.x < 64) {
    uint32_t ea, eb;
    lb_lookback(status, (int)E.c, (int)(o_sf / kTile), ea, eb, diag);
    if (threadIdx.x == 0) {
      s_excl = ea;
      if (sl_cont) lb_publish(status + E.c, 2u, ea + cnt_sl, 0u);
    }
  }
  __syncthreads();
  E.excl_sf = s_excl;
}

// Position inside segment l's list of the flagged element at chunk offset x.
__device__ __forceinline__ uint32_t list_pos(const Tables& T, const EmitCtx& E, const uint32_t* gp, int l,
                                             uint32_t x_prefix, uint32_t total) {
  if (E.sf == E.sl) return E.excl_sf + x_prefix;
  const uint32_t o = (uint32_t)T.seg_off[l];
  const uint32_t start = max(o, E.lo);
  const uint32_t sp = chunk_prefix(gp, start - E.lo, kTile / 4, total);
  return (l == E.sf ? E.excl_sf : 0u) + x_prefix - sp;
}

// Count of flagged elements of segment l inside the chunk.
__device__ __forceinline__ uint32_t chunk_count(const Tables& T, const EmitCtx& E, const uint32_t* gp, int l,
                                                uint32_t total) {
  const uint32_t o = (uint32_t)T.seg_off[l], e = (uint32_t)T.seg_off[l + 1];
  const uint32_t a = max(o, E.lo), b = min(e, E.hi);
  return chunk_prefix(gp, b - E.lo, kTile / 4, total) - chunk_prefix(gp, a - E.lo, kTile / 4, total);
}

// ---------------------------------------------------------------------------------------------
// Top-k level 0: fused accumulate + histogram of bits 30:20 of the magnitude key.
// ---------------------------------------------------------------------------------------------
template <int GDT, bool FUSED>
__global__ __launch_bounds__(kNT) void k_topk_hist(Tables T, const void* g, const float* src, float* acc_out,
                                                   WS ws) {
  __shared__ uint32_t hist[kHBins];
  __shared__ uint32_t lds[kWaves];
  const uint32_t c = blockIdx.x;
  const uint32_t lo = c * kTile, hi = min((uint32_t)T.d, lo + kTile);
  const int sf = T.chunk_sf[c], sl = T.chunk_sl[c];
  const bool uni = sf == sl;
  for (int b = threadIdx.x; b < kHBins; b += kNT) hist[b] = 0;
  __syncthreads();
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t i0 = lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    if (i0 >= hi) break;
    const int nv = (int)min(4u, hi - i0);
    float a[4];
    if constexpr (FUSED) {
      float gv[4], ev[4];
      load4g<GDT>(g, i0, nv, gv);
      load4(src, i0, nv, ev);
#pragma unroll
      for (int q = 0; q < 4; ++q) a[q] = gv[q] + ev[q];
      store4(acc_out, i0, nv, a);
    } else {
      load4(src, i0, nv, a);
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (q < nv) {
        const uint32_t bin = mag_key(a[q]) >> 20;
        if (uni) {
          atomicAdd(&hist[bin], 1u);
        } else {
          const int l = seg_of(i0 + q, sf, sl, T.seg_off);
          atomicAdd(hist_row(ws, 0, T.L, l) + bin, 1u);
        }
      }
    }
  }
  __syncthreads();
  if (uni) {
    uint32_t* row = hist_row(ws, 0, T.L, sf);
    for (int b = threadIdx.x; b < kHBins; b += kNT) {
      const uint32_t v = hist[b];
      if (v) atomicAdd(row + b, v);
    }
  }
  arrive_and_resolve(ws.arrive, T.seg_nchunks, sf, sl, [&](int l) {
    const uint32_t need = (uint32_t)T.seg_k[l];
    const uint32_t* row = hist_row(ws, 0, T.L, l);
    uint32_t above;
    int bin = block_resolve<true>(row, kHBins, need, lds, above);
    if (threadIdx.x == 0) {
      uint32_t* R = res_of(ws, l);
      if (bin < 0) {  // cannot happen: the row holds all d_l >= k_l elements
        atomicOr(ws.diag, kDiagSpinTimeout);
        bin = 0;
      }
      const uint32_t nb = ld_acq(row + bin);
      const uint32_t cnt = above + nb;
      const uint32_t cap = (uint32_t)(T.tk_base[l + 1] - T.tk_base[l]);
      R[R_PREFIX] = (uint32_t)bin << 20;
      R[R_KNOWN] = 12;
      R[R_NEED] = need - above;
      R[R_ABOVE0] = above;
      R[R_CNT] = cnt;
      R[R_SLOW] = cnt > cap ? 1u : 0u;
      if (cnt > cap) atomicOr(ws.diag, kDiagSlowPath);
    }
  });
}

// ---------------------------------------------------------------------------------------------
// Top-k level 1: emit every element whose key is at or above the level-0 bin into the
// segment's list (index order) and histogram bits 19:10 of those inside the bin.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(kNT) void k_topk_emit(Tables T, const float* acc, WS ws) {
  __shared__ uint32_t gp[kTile / 4];
  __shared__ uint32_t lds[kWaves];
  __shared__ uint32_t s_c;
  if (threadIdx.x == 0) s_c = atomicAdd(ws.tickets + 0, 1u);
  __syncthreads();
  EmitCtx E;
  E.c = s_c;
  E.lo = E.c * kTile;
  E.hi = min((uint32_t)T.d, E.lo + kTile);
  E.sf = T.chunk_sf[E.c];
  E.sl = T.chunk_sl[E.c];
  const bool uni = E.sf == E.sl;
  uint32_t thr_u = 0, slow_u = 1;
  if (uni) {
    const uint32_t* R = res_of(ws, E.sf);
    thr_u = R[R_PREFIX];
    slow_u = R[R_SLOW];
  }
  float v[kRounds][4];
  uint32_t mask[kRounds], gpre[kRounds];
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t i0 = E.lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    const int nv = i0 < E.hi ? (int)min(4u, E.hi - i0) : 0;
    mask[r] = 0;
    if (nv > 0) load4(acc, i0, nv, v[r]);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (q < nv) {
        uint32_t thr = thr_u, slow = slow_u;
        if (!uni) {
          const uint32_t* R = res_of(ws, seg_of(i0 + q, E.sf, E.sl, T.seg_off));
          thr = R[R_PREFIX];
          slow = R[R_SLOW];
        }
        if (!slow && mag_key(v[r][q]) >= thr) mask[r] |= 1u << q;
      }
    }
  }
  uint32_t total;
  ordered_positions(T, ws.st_stream, ws.diag, E, mask, gpre, gp, lds, total);
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    if (!mask[r]) continue;
    const uint32_t i0 = E.lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    uint32_t pre = gpre[r];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (mask[r] & (1u << q)) {
        const uint32_t i = i0 + q;
        const int l = uni ? E.sf : seg_of(i, E.sf, E.sl, T.seg_off);
        const uint32_t pos = list_pos(T, E, gp, l, pre, total);
        const uint32_t at = (uint32_t)T.tk_base[l] + pos;
        if (at < (uint32_t)T.tk_base[l + 1]) {
          ws.list_idx[at] = i;
          ws.list_val[at] = v[r][q];
        }
        const uint32_t key = mag_key(v[r][q]);
        const uint32_t* R = res_of(ws, l);
        if ((key >> 20) == (R[R_PREFIX] >> 20)) atomicAdd(hist_row(ws, 1, T.L, l) + ((key >> 10) & 1023u), 1u);
        ++pre;
      }
    }
  }
  arrive_and_resolve(ws.arrive + T.L, T.seg_nchunks, E.sf, E.sl, [&](int l) {
    uint32_t* R = res_of(ws, l);
    if (R[R_SLOW]) return;
    uint32_t above;
    const int bin = block_resolve<true>(hist_row(ws, 1, T.L, l), 1024, R[R_NEED], lds, above);
    if (threadIdx.x == 0) {
      R[R_PREFIX] |= (uint32_t)max(bin, 0) << 10;
      R[R_KNOWN] = 22;
      R[R_NEED] -= above;
    }
  });
}

// ---------------------------------------------------------------------------------------------
// Random-k candidate pass: acc = g + e (written to e when fused), Philox key per element; keys
// below the segment's bound tau are emitted to the list in index order, and the first level of
// the key histogram is built.  The chunk completing a segment checks the candidate count and
// resolves that level.
// ---------------------------------------------------------------------------------------------
template <int GDT, bool FUSED>
__global__ __launch_bounds__(kNT) void k_randk_stream(Tables T, const void* g, const float* src, float* acc_out,
                                                      uint32_t s0, uint32_t s1, uint32_t step, WS ws) {
  __shared__ uint32_t gp[kTile / 4];
  __shared__ uint32_t lds[kWaves];
  __shared__ uint32_t s_c;
  if (threadIdx.x == 0) s_c = atomicAdd(ws.tickets + 0, 1u);
  __syncthreads();
  EmitCtx E;
  E.c = s_c;
  E.lo = E.c * kTile;
  E.hi = min((uint32_t)T.d, E.lo + kTile);
  E.sf = T.chunk_sf[E.c];
  E.sl = T.chunk_sl[E.c];
  const bool uni = E.sf == E.sl;
  const uint32_t o_u = (uint32_t)T.seg_off[E.sf];
  const uint64_t tau_u = T.seg_tau[E.sf];
  const bool aligned = uni && (o_u & 3u) == 0;
  float v[kRounds][4];
  uint32_t key[kRounds][4];
  uint32_t mask[kRounds], gpre[kRounds];
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    const uint32_t i0 = E.lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    const int nv = i0 < E.hi ? (int)min(4u, E.hi - i0) : 0;
    mask[r] = 0;
    if (nv > 0) {
      if constexpr (FUSED) {
        float gv[4], ev[4];
        load4g<GDT>(g, i0, nv, gv);
        load4(src, i0, nv, ev);
#pragma unroll
        for (int q = 0; q < 4; ++q) v[r][q] = gv[q] + ev[q];
        store4(acc_out, i0, nv, v[r]);
      } else {
        load4(src, i0, nv, v[r]);
      }
      if (aligned) {
        const uint4 x = philox(make_uint4((i0 - o_u) >> 2, 0u, step, kRandkTag | (uint32_t)E.sf), s0, s1);
        key[r][0] = x.x; key[r][1] = x.y; key[r][2] = x.z; key[r][3] = x.w;
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (q < nv && (uint64_t)key[r][q] < tau_u) mask[r] |= 1u << q;
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          key[r][q] = 0;
          if (q < nv) {
            const uint32_t i = i0 + q;
            const int l = uni ? E.sf : seg_of(i, E.sf, E.sl, T.seg_off);
            key[r][q] = randk_key(i - (uint32_t)T.seg_off[l], (uint32_t)l, step, s0, s1);
            if ((uint64_t)key[r][q] < T.seg_tau[l]) mask[r] |= 1u << q;
          }
        }
      }
    }
  }
  uint32_t total;
  ordered_positions(T, ws.st_stream, ws.diag, E, mask, gpre, gp, lds, total);
#pragma unroll
  for (int r = 0; r < kRounds; ++r) {
    if (!mask[r]) continue;
    const uint32_t i0 = E.lo + (uint32_t)(r * kNT + threadIdx.x) * 4u;
    uint32_t pre = gpre[r];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (mask[r] & (1u << q)) {
        const uint32_t i = i0 + q;
        const int l = uni ? E.sf : seg_of(i, E.sf, E.sl, T.seg_off);
        const uint32_t pos = list_pos(T, E, gp, l, pre, total);
        const uint32_t cap = (uint32_t)(T.rk_base[l + 1] - T.rk_base[l]);
        if (pos < cap) {
          const uint32_t at = (uint32_t)T.rk_base[l] + pos;
          ws.list_idx[at] = i;
          ws.list_val[at] = v[r][q];
          ws.list_key[at] = key[r][q];
        }
        const int hb = T.seg_hb[l];
        const int w = min(11, hb);
        const uint32_t kk = ~key[r][q];
        atomicAdd(hist_row(ws, 0, T.L, l) + ((kk >> (hb - w)) & ((1u << w) - 1u)), 1u);
        ++pre;
      }
    }
  }
  // per-segment candidate counts
  for (int l = E.sf + (int)threadIdx.x; l <= E.sl; l += kNT) {
    const uint32_t n = chunk_count(T, E, gp, l, total);
    if (n) atomicAdd(ws.cnt + l, n);
  }
  arrive_and_resolve(ws.arrive, T.seg_nchunks, E.sf, E.sl, [&](int l) {
    uint32_t* R = res_of(ws, l);
    const uint32_t cnt = ld_acq(ws.cnt + l);
    const uint32_t k = (uint32_t)T.seg_k[l];
    const uint32_t cap = (uint32_t)(T.rk_base[l + 1] - T.rk_base[l]);
    const int hb = T.seg_hb[l];
    const int w = min(11, hb);
    if (cnt < k || cnt > cap) {
      if (threadIdx.x == 0) {
        R[R_SLOW] = 1;
        R[R_CNT] = 0;
        atomicOr(ws.diag, kDiagSlowPath);
      }
      return;
    }
    uint32_t above;
    const int bin = block_resolve<true>(hist_row(ws, 0, T.L, l), 1 << w, k, lds, above);
    if (threadIdx.x == 0) {
      const uint32_t top = hb >= 32 ? 0u : (0xFFFFFFFFu << hb);
      R[R_PREFIX] = top | ((uint32_t)max(bin, 0) << (hb - w));
      R[R_KNOWN] = (uint32_t)(32 - hb + w);
      R[R_NEED] = k - above;
      R[R_CNT] = cnt;
      R[R_SLOW] = 0;
    }
  });
}

// ---------------------------------------------------------------------------------------------
// List selection: next radix level over the candidate lists, and the exact slow path.
// KIND 0 = top-k (key = magnitude bits of the value), 1 = random-k (key = ~Philox key, so the
// smallest random keys rank highest).  Ties between equal keys go to the lower list position,
// which is the lower element index.
// ---------------------------------------------------------------------------------------------
template <int KIND>
__device__ __forceinline__ uint32_t list_key_of(const WS& ws, uint32_t p) {
  if constexpr (KIND == 0) return mag_key(ws.list_val[p]);
  else return ~ws.list_key[p];
}

struct ListGeom {
  const int32_t* base;
  const int32_t* nlch;
  const int32_t* lsf;
  const int32_t* lsl;
  uint32_t nlchunks;
};

template <int KIND>
__device__ __forceinline__ ListGeom list_geom(const Tables& T) {
  if constexpr (KIND == 0) return ListGeom{T.tk_base, T.tk_nlch, T.tk_lsf, T.tk_lsl, (uint32_t)T.tk_nlchunks};
  else return ListGeom{T.rk_base, T.rk_nlch, T.rk_lsf, T.rk_lsl, (uint32_t)T.rk_nlchunks};
}

// Exact single-workgroup selection over the whole segment (used when the list cannot hold the
// answer).  Radix levels over the keys of all d_l elements, then an index-ordered emission.
template <int KIND>
__device__ void slow_select(const Tables& T, WS& ws, int l, const float* data, float* e_zero,
                            uint32_t* out_idx, float* out_val, uint32_t s0, uint32_t s1, uint32_t step,
                            uint32_t* lhist, uint32_t* lds) {
  uint32_t* R = res_of(ws, l);
  const uint32_t o = (uint32_t)T.seg_off[l], n = (uint32_t)T.seg_off[l + 1] - o;
  const uint32_t P = (uint32_t)T.seg_P[l];
  uint32_t prefix, need;
  int known;
  if constexpr (KIND == 0) {
    prefix = R[R_PREFIX];  // level 0 (bits 31:20) resolved by the histogram pass
    need = R[R_NEED];
    known = 12;
  } else {
    prefix = 0;
    need = (uint32_t)T.seg_k[l];
    known = 0;
  }
  auto keyat = [&](uint32_t j) -> uint32_t {
    if constexpr (KIND == 0) return mag_key(data[o + j]);
    else return ~randk_key(j, (uint32_t)l, step, s0, s1);
  };
  while (known < 32) {
    const int w = min(11, 32 - known);
    const int shift = 32 - known - w;
    for (int b = threadIdx.x; b < (1 << w); b += kNT) lhist[b] = 0;
    __syncthreads();
    for (uint32_t j = threadIdx.x; j < n; j += kNT) {
      const uint32_t k = keyat(j);
      if (known == 0 || (k >> (32 - known)) == (prefix >> (32 - known)))
        atomicAdd(&lhist[(k >> shift) & ((1u << w) - 1u)], 1u);
    }
    __syncthreads();
    uint32_t above;
    const int bin = block_resolve<false>(lhist, 1 << w, need, lds, above);
    prefix |= (uint32_t)max(bin, 0) << shift;
    need -= above;
    known += w;
  }
  const uint32_t Tk = prefix, r = need;
  uint32_t run_a = 0, run_b = 0;
  for (uint32_t j0 = 0; j0 < n; j0 += kNT) {
    const uint32_t j = j0 + threadIdx.x;
    uint32_t a = 0, b = 0, k = 0;
    if (j < n) {
      k = keyat(j);
      a = k > Tk;
      b = k == Tk;
    }
    uint32_t tot;
    const uint32_t ex = block_excl_scan(a | (b << 16), lds, tot);
    const uint32_t ea = run_a + (ex & 0xFFFFu), eb = run_b + (ex >> 16);
    if ((a || (b && eb < r)) && ea + min(eb, r) < (uint32_t)T.seg_k[l]) {
      const uint32_t pos = P + ea + min(eb, r);
      out_idx[pos] = o + j;
      out_val[pos] = data[o + j];
      if (e_zero) e_zero[o + j] = 0.0f;
    }
    run_a += tot & 0xFFFFu;
    run_b += tot >> 16;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    R[R_DONE] = 1;
    R[R_CNT] = 0;
  }
}

template <int KIND>
__global__ __launch_bounds__(kNT) void k_list_level(Tables T, WS ws, int slot, const float* data, float* e_zero,
                                                    uint32_t* out_idx, float* out_val, uint32_t s0, uint32_t s1,
                                                    uint32_t step) {
  __shared__ uint32_t lhist[kHBins];
  __shared__ uint32_t lds[kWaves];
  const ListGeom G = list_geom<KIND>(T);
  const uint32_t q = blockIdx.x;
  const uint32_t lo = q * kLTile;
  const int sf = G.lsf[q], sl = G.lsl[q];
  for (int rr = 0; rr < kLRounds; ++rr) {
    const uint32_t p = lo + (uint32_t)(rr * kNT) + threadIdx.x;
    const int l = sf == sl ? sf : seg_of(p, sf, sl, G.base);
    const uint32_t* R = res_of(ws, l);
    if (p >= (uint32_t)G.base[l + 1] || R[R_SLOW] || R[R_KNOWN] >= 32) continue;
    if (p >= (uint32_t)G.base[l] + R[R_CNT]) continue;
    const uint32_t known = R[R_KNOWN], prefix = R[R_PREFIX];
    const uint32_t k = list_key_of<KIND>(ws, p);
    if ((k >> (32 - known)) != (prefix >> (32 - known))) continue;
    const int w = min(11, 32 - (int)known);
    const int shift = 32 - (int)known - w;
    atomicAdd(hist_row(ws, slot, T.L, l) + ((k >> shift) & ((1u << w) - 1u)), 1u);
  }
  arrive_and_resolve(ws.arrive + (size_t)slot * T.L, G.nlch, sf, sl, [&](int l) {
    uint32_t* R = res_of(ws, l);
    if (R[R_SLOW]) {
      if (!R[R_DONE]) slow_select<KIND>(T, ws, l, data, e_zero, out_idx, out_val, s0, s1, step, lhist, lds);
      return;
    }
    const int known = (int)R[R_KNOWN];
    if (known >= 32) return;
    const int w = min(11, 32 - known);
    const int shift = 32 - known - w;
    uint32_t above;
    const int bin = block_resolve<true>(hist_row(ws, slot, T.L, l), 1 << w, R[R_NEED], lds, above);
    if (threadIdx.x == 0) {
      R[R_PREFIX] |= (uint32_t)max(bin, 0) << shift;
      R[R_KNOWN] = (uint32_t)(known + w);
      R[R_NEED] -= above;
    }
  });
}

// Emission: every list entry with key > T, plus the first r entries with key == T, written in
// list (= index) order to the message; e is zeroed at the sent indices when fused.
template <int KIND>
__global__ __launch_bounds__(kNT) void k_list_emit(Tables T, WS ws, uint32_t* out_idx, float* out_val, float* e_zero) {
  __shared__ uint32_t gp[kLTile];
  __shared__ uint32_t lds[kWaves];
  __shared__ uint32_t s_c, s_ea, s_eb;
  const ListGeom G = list_geom<KIND>(T);
  if (threadIdx.x == 0) s_c = atomicAdd(ws.tickets + 1, 1u);
  __syncthreads();
  const uint32_t q = s_c;
  const uint32_t lo = q * kLTile, hi = lo + kLTile;
  const int sf = G.lsf[q], sl = G.lsl[q];
  const bool uni = sf == sl;
  uint32_t fa[kLRounds], fb[kLRounds], pre[kLRounds];
  uint32_t base = 0;
#pragma unroll
  for (int rr = 0; rr < kLRounds; ++rr) {
    const uint32_t p = lo + (uint32_t)(rr * kNT) + threadIdx.x;
    const int l = uni ? sf : seg_of(p, sf, sl, G.base);
    const uint32_t* R = res_of(ws, l);
    fa[rr] = fb[rr] = 0;
    if (p < (uint32_t)G.base[l + 1] && !R[R_SLOW] && p < (uint32_t)G.base[l] + R[R_CNT]) {
      const uint32_t k = list_key_of<KIND>(ws, p), Tk = R[R_PREFIX];
      fa[rr] = k > Tk;
      fb[rr] = k == Tk;
    }
    uint32_t tot;
    const uint32_t ex = block_excl_scan(fa[rr] | (fb[rr] << 16), lds, tot);
    pre[rr] = base + ex;
    gp[rr * kNT + threadIdx.x] = base + ex;
    base += tot;
  }
  __syncthreads();
  const uint32_t total = base;
  // gp[x] is the packed exclusive prefix at list position lo + x (entry (rr, t) has x = rr*kNT + t).
  auto prefix_at = [&](uint32_t p) -> uint32_t { return p >= hi ? total : gp[p - lo]; };
  const uint32_t b_sl = (uint32_t)G.base[sl];
  const uint32_t st_sl = max(b_sl, lo);
  const uint32_t c_sl = total - prefix_at(st_sl);
  const bool sl_cont = b_sl < lo;
  const uint32_t b_sf = (uint32_t)G.base[sf];
  const bool need_lb = b_sf < lo;
  if (threadIdx.x == 0) {
    lb_publish(ws.st_emit + q, sl_cont ? 1u : 2u, c_sl & 0xFFFFu, c_sl >> 16);
    s_ea = 0;
    s_eb = 0;
  }
  if (need_lb && threadIdx.x < 64) {
    uint32_t ea, eb;
    lb_lookback(ws.st_emit, (int)q, (int)(b_sf / kLTile), ea, eb, ws.diag);
    if (threadIdx.x == 0) {
      s_ea = ea;
      s_eb = eb;
      if (sl_cont) lb_publish(ws.st_emit + q, 2u, ea + (c_sl & 0xFFFFu), eb + (c_sl >> 16));
    }
  }
  __syncthreads();
#pragma unroll
  for (int rr = 0; rr < kLRounds; ++rr) {
    if (!(fa[rr] | fb[rr])) continue;
    const uint32_t p = lo + (uint32_t)(rr * kNT) + threadIdx.x;
    const int l = uni ? sf : seg_of(p, sf, sl, G.base);
    const uint32_t* R = res_of(ws, l);
    uint32_t a, b;
    if (uni) {
      a = s_ea + (pre[rr] & 0xFFFFu);
      b = s_eb + (pre[rr] >> 16);
    } else {
      const uint32_t sp = prefix_at(max((uint32_t)G.base[l], lo));
      a = (l == sf ? s_ea : 0u) + (pre[rr] & 0xFFFFu) - (sp & 0xFFFFu);
      b = (l == sf ? s_eb : 0u) + (pre[rr] >> 16) - (sp >> 16);
    }
    const uint32_t r = R[R_NEED];
    if ((fa[rr] || b < r) && a + min(b, r) < (uint32_t)T.seg_k[l]) {
      const uint32_t pos = (uint32_t)T.seg_P[l] + a + min(b, r);
      const uint32_t i = ws.list_idx[p];
      out_idx[pos] = i;
      out_val[pos] = ws.list_val[p];
      if (e_zero && i < (uint32_t)T.d) e_zero[i] = 0.0f;
    }
  }
}

}  // namespace efs
