// Device-side building blocks for the efsparse kernels (gfx950, wave64).
//
// Philox4x32-10 (Salmon et al., SC 2011), magnitude keys, streaming loads and stores,
// wave / workgroup scans and a histogram resolve used by the radix selections.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace efs {

constexpr int kNT = 256;                      // threads per workgroup of most kernels
constexpr int kSelNT = 1024;                  // threads per workgroup of the per-segment kernels
constexpr uint32_t kTile = 4096;              // data elements per tile (the rows of the selection kernels)
constexpr int kHBins = 2048;                  // LDS histogram bins (11 bits per radix level)
constexpr int kResWords = 16;                // per-segment selection record (uint32 words)
constexpr int kSubLists = 16;                // a segment's list of undecided candidates is kept as 16
                                              // sub-lists (row r appends to sub-list r % 16)
constexpr int kSampleMax = 32768;             // top-k threshold sample size (keys held in LDS)
constexpr int kExactMax = 4096;               // top-k: segments up to this size are sampled whole (exact rule)
constexpr int kSampleRun = 256;               // samples per sample run (one workgroup each)
constexpr int kSampleTotal = 16384;           // top-k: samples shared by a layout's sampled segments
constexpr int kSampleCap = 65536;             // ... or this many where the margin would hold many candidates
constexpr int kSampleMinRuns = 4;             // top-k: at least this many runs per sampled segment

constexpr uint32_t kRandkTag = 0x01000000u;
constexpr uint32_t kRandblockTag = 0x02000000u;
constexpr uint32_t kSampleTag = 0x03000000u;  // top-k: positions of the threshold sample

constexpr uint32_t kDiagSlowPath = 2u;
constexpr uint32_t kDiagRetry = 8u;  // a top-k segment re-collected its candidates at a lower threshold

// Per-segment selection record, uint32 words.  Key' is the selection key (top-k: magnitude bits;
// random-k: complement of the Philox key), larger is better; among equal key' the lower index wins.
enum : int {
  R_A = 0,      // candidates: key' > R_A, or key' == R_A with index < R_IA
  R_IA = 1,
  R_T = 2,      // winners: key' > R_T, or key' == R_T with index < R_IT
  R_IT = 3,
  R_SLOW = 4,   // 1: the candidates cannot hold the answer; the segment is resolved over all of
                //    its elements
  R_MODE = 5,   // 1: the candidates are exactly the winners (threshold from the whole segment)
  R_SH = 6,     // candidate histogram: bin shift
  R_B = 7,      // candidate histogram: bin holding the k_l-th best candidate
  R_NEED = 8,   // winners still needed from bin R_B (retry: from the listed candidates)
  R_RETRY = 9,  // top-k: 1 when the segment's candidates fell short of k_l and are collected again
  R_A2 = 10,    // top-k retry: the lower threshold; keys in (R_A2, R_A) are the listed candidates,
                //   keys equal to it are counted
  R_OVF = 11,   // top-k: candidates did not fit the workspace (a retry collects them again, else the
                //   exact path runs)
};

constexpr int kBtWords = 8;  // words per record of the block aggregate's (tile, segment) table

struct Tables {
  const int32_t* seg_off;      // [L+1]
  const int32_t* seg_k;        // [L]
  const int32_t* seg_P;        // [L+1]
  const int32_t* seg_bl;       // [L]
  const int32_t* seg_nb;       // [L]
  const int32_t* seg_srank;    // [L]   top-k: rank of the candidate threshold inside the sample
  const int32_t* seg_urank;    // [L]   top-k: sample rank bounding the k-th key from above
  const int32_t* seg_cbase;    // [L+1] first row of each segment (a row = segment x data tile)
  const int32_t* seg_ro;       // [L+1] first top-k sample run of each segment
  const uint64_t* seg_tau;     // [L]   random-k: Philox keys below tau are candidates
  const uint32_t* seg_ulo;     // [L]   random-k: keys below ulo are winners if at most k_l are
  const uint64_t* seg_lbase;   // [L]   first entry of the segment's list region in the list arrays
  const uint32_t* seg_lq;      // [L]   entries per sub-list in that region (min(kSubLists, rows) sub-lists)
  const uint32_t* seg_zc;      // [L]   top-k: 1 when the fused pass stores +0 at the candidates
  const int32_t* chunk_sf;     // [nchunks] first / last segment of each data tile
  const int32_t* chunk_sl;
  const int32_t* row_seg;      // [nrows] segment of each row
  const int32_t* run_seg;      // [nruns] top-k: segment of each sample run
  const uint32_t* row_rec;     // [4 nrows] multi-segment layouts: per row its segment, the
                               // segment's offset and end, and the row's tile base
  const uint32_t* btile;       // [kBtWords nbtiles] block aggregate, multi-segment layouts: for every
                               // (1024-element data tile, segment) pair with an element in common:
                               // tile, segment, its offset, size, k and message offset, 0, 0
  int32_t d, L, nchunks, nrows, nruns, nbtiles;
  int32_t K;                   // the sum of the k_l (one segment: its k)
  int32_t rk_direct;           // random-k: k_stream_sel counts the certain winners and lists the
                               // undecided candidates of every row; k_select gathers the lists
  int32_t tk_retry;            // top-k: the candidate retry is enabled
};

// ---------------------------------------------------------------------------------------------
// Philox4x32-10: 10 rounds; each multiplies words 0 and 2 by fixed constants, keeps both product
// halves and mixes the high halves with words 1, 3 and the round key; the key advances by two
// Weyl constants between rounds.
// ---------------------------------------------------------------------------------------------
__device__ __forceinline__ uint4 philox(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
    c = make_uint4((uint32_t)(p1 >> 32) ^ c.y ^ k0, (uint32_t)p1, (uint32_t)(p0 >> 32) ^ c.w ^ k1,
                   (uint32_t)p0);
  }
  return c;
}

__device__ __forceinline__ uint32_t word(const uint4& v, int q) {
  return q == 0 ? v.x : q == 1 ? v.y : q == 2 ? v.z : v.w;
}

// Random-k key of local position j in segment l.
__device__ __forceinline__ uint32_t randk_key(uint32_t j, uint32_t l, uint32_t step, uint32_t s0,
                                              uint32_t s1) {
  uint4 x = philox(make_uint4(j >> 2, 0u, step, kRandkTag | l), s0, s1);
  return word(x, j & 3);
}

// Random-block start of segment l (segment-local).
__device__ __forceinline__ uint32_t block_start(uint32_t l, uint32_t step, uint32_t s0, uint32_t s1,
                                                uint32_t bl, uint32_t nb) {
  uint4 x = philox(make_uint4(0u, 0u, step, kRandblockTag | l), s0, s1);
  const uint64_t r = (uint64_t)x.x | ((uint64_t)x.y << 32);
  return bl * (uint32_t)__umul64hi(r, (uint64_t)nb);
}

__device__ __forceinline__ uint32_t mag_key(float x) { return __float_as_uint(x) & 0x7FFFFFFFu; }

// ---------------------------------------------------------------------------------------------
// Memory helpers.  The streaming passes touch each byte once, so their loads and stores carry the
// nontemporal hint.
// ---------------------------------------------------------------------------------------------
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u2v __attribute__((ext_vector_type(2)));

__device__ __forceinline__ void load4(const float* p, uint32_t i0, int nv, float v[4]) {
  if (nv == 4) {
    const f4 x = __builtin_nontemporal_load(reinterpret_cast<const f4*>(p + i0));
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = q < nv ? p[i0 + q] : 0.0f;
  }
}

__device__ __forceinline__ float bf16_to_f32(uint32_t b) { return __uint_as_float(b << 16); }

template <int GDT>
__device__ __forceinline__ void load4g(const void* g, uint32_t i0, int nv, float v[4]) {
  if constexpr (GDT == 0) {
    load4(reinterpret_cast<const float*>(g), i0, nv, v);
  } else {
    const uint16_t* p = reinterpret_cast<const uint16_t*>(g);
    if (nv == 4) {
      const u2v x = __builtin_nontemporal_load(reinterpret_cast<const u2v*>(p + i0));
      v[0] = bf16_to_f32(x.x & 0xFFFFu); v[1] = bf16_to_f32(x.x >> 16);
      v[2] = bf16_to_f32(x.y & 0xFFFFu); v[3] = bf16_to_f32(x.y >> 16);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = q < nv ? bf16_to_f32(p[i0 + q]) : 0.0f;
    }
  }
}

template <int GDT>
__device__ __forceinline__ float load1g(const void* g, uint32_t i) {
  if constexpr (GDT == 0) return reinterpret_cast<const float*>(g)[i];
  else return bf16_to_f32(reinterpret_cast<const uint16_t*>(g)[i]);
}

__device__ __forceinline__ void store4(float* p, uint32_t i0, int nv, const float v[4]) {
  if (nv == 4) {
    const f4 x = {v[0], v[1], v[2], v[3]};
    __builtin_nontemporal_store(x, reinterpret_cast<f4*>(p + i0));
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (q < nv) p[i0 + q] = v[q];
  }
}

// Unconditional variants for groups known to be whole.  Keeping the masked forms (which branch
// on the group's extent) out of the common path lets every load of a thread be issued before
// the first wait.
__device__ __forceinline__ void load4f(const float* p, uint32_t i0, float v[4]) {
  const f4 x = __builtin_nontemporal_load(reinterpret_cast<const f4*>(p + i0));
  v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
}

template <int GDT>
__device__ __forceinline__ void load4gf(const void* g, uint32_t i0, float v[4]) {
  if constexpr (GDT == 0) {
    load4f(reinterpret_cast<const float*>(g), i0, v);
  } else {
    const u2v x = __builtin_nontemporal_load(reinterpret_cast<const u2v*>(reinterpret_cast<const uint16_t*>(g) + i0));
    v[0] = bf16_to_f32(x.x & 0xFFFFu); v[1] = bf16_to_f32(x.x >> 16);
    v[2] = bf16_to_f32(x.y & 0xFFFFu); v[3] = bf16_to_f32(x.y >> 16);
  }
}

// Masked variants: vm has bit q set when element i0 + q is inside the row being processed.
__device__ __forceinline__ uint32_t group_mask(uint32_t i0, uint32_t lo, uint32_t hi) {
  uint32_t m = 0;
#pragma unroll
  for (int q = 0; q < 4; ++q)
    if (i0 + q >= lo && i0 + q < hi) m |= 1u << q;
  return m;
}

__device__ __forceinline__ void load4m(const float* p, uint32_t i0, uint32_t vm, float v[4]) {
  if (vm == 0xFu) {
    const f4 x = __builtin_nontemporal_load(reinterpret_cast<const f4*>(p + i0));
    v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = (vm >> q) & 1u ? p[i0 + q] : 0.0f;
  }
}

template <int GDT>
__device__ __forceinline__ void load4gm(const void* g, uint32_t i0, uint32_t vm, float v[4]) {
  if constexpr (GDT == 0) {
    load4m(reinterpret_cast<const float*>(g), i0, vm, v);
  } else {
    const uint16_t* p = reinterpret_cast<const uint16_t*>(g);
    if (vm == 0xFu) {
      const u2v x = __builtin_nontemporal_load(reinterpret_cast<const u2v*>(p + i0));
      v[0] = bf16_to_f32(x.x & 0xFFFFu); v[1] = bf16_to_f32(x.x >> 16);
      v[2] = bf16_to_f32(x.y & 0xFFFFu); v[3] = bf16_to_f32(x.y >> 16);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = (vm >> q) & 1u ? bf16_to_f32(p[i0 + q]) : 0.0f;
    }
  }
}

__device__ __forceinline__ void store4m(float* p, uint32_t i0, uint32_t vm, const float v[4]) {
  if (vm == 0xFu) {
    const f4 x = {v[0], v[1], v[2], v[3]};
    __builtin_nontemporal_store(x, reinterpret_cast<f4*>(p + i0));
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if ((vm >> q) & 1u) p[i0 + q] = v[q];
  }
}

// Segment containing element i, searching segments [sf, sl] (sf <= answer <= sl).
__device__ __forceinline__ int seg_of(uint32_t i, int sf, int sl, const int32_t* off) {
  while (sf < sl) {
    const int mid = (sf + sl + 1) >> 1;
    if ((uint32_t)off[mid] <= i) sf = mid; else sl = mid - 1;
  }
  return sf;
}

// First position j in [0, n) with a[j] >= x (a ascending), n if none.
__device__ __forceinline__ uint32_t lower_bound_u32(const uint32_t* a, uint32_t n, uint32_t x) {
  uint32_t lo = 0, hi = n;
  while (lo < hi) {
    const uint32_t mid = (lo + hi) >> 1;
    if (a[mid] < x) lo = mid + 1; else hi = mid;
  }
  return lo;
}

__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// ---------------------------------------------------------------------------------------------
// Scans
// ---------------------------------------------------------------------------------------------
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t n = __shfl_up(v, o, 64);
    if (lane >= o) v += n;
  }
  return v;
}

// Exclusive scan over the workgroup (NT threads) in thread order; `lds` holds NT/64 words.  Two
// 16-bit counters can be packed into v as long as workgroup totals stay below 65536.
template <int NT>
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* lds, uint32_t& total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const uint32_t inc = wave_incl_scan(v);
  if (lane == 63) lds[wid] = inc;
  __syncthreads();
  uint32_t off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < NT / 64; ++w) {
    const uint32_t x = lds[w];
    off += (w < wid) ? x : 0u;
    tot += x;
  }
  __syncthreads();
  total = tot;
  return off + inc - v;
}

// Exclusive scans of NV counters at once (one pair of barriers); `lds` holds NV * NT/64 words.
template <int NT, int NV>
__device__ __forceinline__ void block_excl_scan_n(const uint32_t (&v)[NV], uint32_t* lds, uint32_t (&ex)[NV],
                                                  uint32_t (&total)[NV]) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  uint32_t inc[NV];
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    inc[j] = wave_incl_scan(v[j]);
    if (lane == 63) lds[j * (NT / 64) + wid] = inc[j];
  }
  __syncthreads();
#pragma unroll
  for (int j = 0; j < NV; ++j) {
    uint32_t off = 0, tot = 0;
#pragma unroll
    for (int w = 0; w < NT / 64; ++w) {
      const uint32_t x = lds[j * (NT / 64) + w];
      off += (w < wid) ? x : 0u;
      tot += x;
    }
    ex[j] = off + inc[j] - v[j];
    total[j] = tot;
  }
  __syncthreads();
}

// Scanning an LDS histogram from its highest bin down, find the bin in which the running count
// reaches `need`.  Returns the bin (-1 if the histogram holds fewer than `need`) and, through
// `above`, the count in strictly higher bins.  Every thread gets the result.
template <int NT>
__device__ __forceinline__ int block_resolve(const uint32_t* hist, int nb, uint32_t need, uint32_t* lds, uint32_t& above) {
  __shared__ int s_bin;
  __shared__ uint32_t s_above;
  constexpr int kMaxPer = (kHBins + NT - 1) / NT;
  const int per = (nb + NT - 1) / NT;
  const int top = nb - 1 - per * (int)threadIdx.x;
  uint32_t h[kMaxPer];
  uint32_t local = 0;
#pragma unroll
  for (int j = 0; j < kMaxPer; ++j) {
    const int b = top - j;
    h[j] = (j < per && b >= 0) ? hist[b] : 0u;
    local += h[j];
  }
  if (threadIdx.x == 0) {
    s_bin = -1;
    s_above = 0;
  }
  uint32_t total;
  const uint32_t excl = block_excl_scan<NT>(local, lds, total);
  if (excl < need && need <= excl + local) {
    uint32_t run = excl;
#pragma unroll
    for (int j = 0; j < kMaxPer; ++j) {
      if (j < per && run + h[j] >= need) {
        s_bin = top - j;
        s_above = run;
        break;
      }
      run += h[j];
    }
  }
  __syncthreads();
  above = s_above;
  const int bin = s_bin;
  __syncthreads();
  return bin;
}

// block_resolve for two counts at once (one scan of the histogram): the bins where the running
// count from the top reaches need_a and need_b (a need of 0 finds nothing: bin -1).
template <int NT>
__device__ __forceinline__ void block_resolve2(const uint32_t* hist, int nb, uint32_t need_a, uint32_t need_b,
                                               uint32_t* lds, int& bin_a, uint32_t& above_a, int& bin_b,
                                               uint32_t& above_b) {
  __shared__ int s_bin2[2];
  __shared__ uint32_t s_above2[2];
  constexpr int kMaxPer = (kHBins + NT - 1) / NT;
  const int per = (nb + NT - 1) / NT;
  const int top = nb - 1 - per * (int)threadIdx.x;
  uint32_t h[kMaxPer];
  uint32_t local = 0;
#pragma unroll
  for (int j = 0; j < kMaxPer; ++j) {
    const int b = top - j;
    h[j] = (j < per && b >= 0) ? hist[b] : 0u;
    local += h[j];
  }
  if (threadIdx.x == 0) {
    s_bin2[0] = s_bin2[1] = -1;
    s_above2[0] = s_above2[1] = 0;
  }
  uint32_t total;
  const uint32_t excl = block_excl_scan<NT>(local, lds, total);
#pragma unroll
  for (int q = 0; q < 2; ++q) {
    const uint32_t need = q == 0 ? need_a : need_b;
    if (excl < need && need <= excl + local) {
      uint32_t run = excl;
#pragma unroll
      for (int j = 0; j < kMaxPer; ++j) {
        if (j < per && run + h[j] >= need) {
          s_bin2[q] = top - j;
          s_above2[q] = run;
          break;
        }
        run += h[j];
      }
    }
  }
  __syncthreads();
  bin_a = s_bin2[0];
  above_a = s_above2[0];
  bin_b = s_bin2[1];
  above_b = s_above2[1];
  __syncthreads();
}

}  // namespace efs
