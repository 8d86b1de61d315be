// Device-side building blocks for the efsparse kernels (gfx950, wave64).
//
// Philox4x32-10 (Salmon et al., SC 2011), magnitude keys, wave/block scans,
// per-segment histogram resolution and a decoupled look-back for ordered
// compaction across workgroups.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace efs {

constexpr int kNT = 256;                      // threads per workgroup
constexpr int kWaves = kNT / 64;
constexpr uint32_t kTile = 8192;              // data elements per chunk
constexpr int kRounds = kTile / (4 * kNT);    // float4 groups per thread per chunk
constexpr uint32_t kLTile = 2048;             // list entries per list chunk
constexpr int kLRounds = kLTile / kNT;
constexpr int kHBins = 2048;                  // histogram row width per segment and level
constexpr int kResWords = 16;                 // per-segment selection record (uint32 words)

constexpr uint32_t kRandkTag = 0x01000000u;
constexpr uint32_t kRandblockTag = 0x02000000u;

// diagnostics bits
constexpr uint32_t kDiagSpinTimeout = 1u;
constexpr uint32_t kDiagSlowPath = 2u;
constexpr int kSpinLimit = 1 << 21;

// Per-segment selection record, uint32 words.
enum : int {
  R_PREFIX = 0,   // known high bits of the threshold key
  R_KNOWN = 1,    // number of known high bits (32 = threshold fully resolved)
  R_NEED = 2,     // entries still to take among those matching the prefix
  R_CNT = 3,      // list entries produced for the segment
  R_SLOW = 4,     // 1: resolved by the exact slow path instead of the list
  R_ABOVE0 = 5,   // top-k: elements above the level-0 bin
  R_DONE = 6,     // 1: output already written (slow path)
};

struct Tables {
  const int32_t* seg_off;      // [L+1]
  const int32_t* seg_k;        // [L]
  const int32_t* seg_P;        // [L+1]
  const int32_t* seg_bl;       // [L]
  const int32_t* seg_nb;       // [L]
  const int32_t* seg_hb;       // [L]  random-k: candidate keys are < 2^hb
  const int32_t* seg_nchunks;  // [L]  data chunks touching the segment
  const uint64_t* seg_tau;     // [L]  random-k: keys below tau are candidates
  const int32_t* tk_base;      // [L+1] top-k list region starts
  const int32_t* tk_nlch;      // [L]  top-k list chunks touching the segment's region
  const int32_t* rk_base;      // [L+1]
  const int32_t* rk_nlch;      // [L]
  const int32_t* chunk_sf;     // [nchunks] first / last segment of each data chunk
  const int32_t* chunk_sl;
  const int32_t* tk_lsf;       // [tk_nlchunks] first / last segment of each top-k list chunk
  const int32_t* tk_lsl;
  const int32_t* rk_lsf;
  const int32_t* rk_lsl;
  int32_t d, L, nchunks, tk_nlchunks, rk_nlchunks, pad;
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
// Memory helpers
// ---------------------------------------------------------------------------------------------
typedef float f4 __attribute__((ext_vector_type(4)));
typedef uint32_t u2v __attribute__((ext_vector_type(2)));

__device__ __forceinline__ void load4(const float* p, uint32_t i0, int nv, float v[4]) {
  if (nv == 4) {
    f4 x = *reinterpret_cast<const f4*>(p + i0);
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
      u2v x = *reinterpret_cast<const u2v*>(p + i0);
      v[0] = bf16_to_f32(x.x & 0xFFFFu); v[1] = bf16_to_f32(x.x >> 16);
      v[2] = bf16_to_f32(x.y & 0xFFFFu); v[3] = bf16_to_f32(x.y >> 16);
    } else {
#pragma unroll
      for (int q = 0; q < 4; ++q) v[q] = q < nv ? bf16_to_f32(p[i0 + q]) : 0.0f;
    }
  }
}

__device__ __forceinline__ void store4(float* p, uint32_t i0, int nv, const float v[4]) {
  if (nv == 4) {
    f4 x = {v[0], v[1], v[2], v[3]};
    *reinterpret_cast<f4*>(p + i0) = x;
  } else {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (q < nv) p[i0 + q] = v[q];
  }
}

__device__ __forceinline__ uint32_t ld_acq(const uint32_t* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Segment containing element i, searching segments [sf, sl] (sf <= answer <= sl).
__device__ __forceinline__ int seg_of(uint32_t i, int sf, int sl, const int32_t* off) {
  while (sf < sl) {
    const int mid = (sf + sl + 1) >> 1;
    if ((uint32_t)off[mid] <= i) sf = mid; else sl = mid - 1;
  }
  return sf;
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

__device__ __forceinline__ uint32_t wave_sum(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Exclusive scan over the workgroup in thread order; `lds` holds kWaves words.
// Two 16-bit counters can be packed into v as long as block totals stay < 65536.
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t v, uint32_t* lds, uint32_t& total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const uint32_t inc = wave_incl_scan(v);
  if (lane == 63) lds[wid] = inc;
  __syncthreads();
  uint32_t off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const uint32_t x = lds[w];
    off += (w < wid) ? x : 0u;
    tot += x;
  }
  __syncthreads();
  total = tot;
  return off + inc - v;
}

// Scanning a histogram from its highest bin down, find the bin in which the running count
// reaches `need`.  Returns the bin (or -1 if the histogram holds fewer than `need` entries) and,
// through `above`, the count in strictly higher bins.  All threads get the result.
template <bool GLOBAL>
__device__ int block_resolve(const uint32_t* hist, int nb, uint32_t need, uint32_t* lds,
                             uint32_t& above) {
  __shared__ int s_bin;
  __shared__ uint32_t s_above;
  const int per = (nb + kNT - 1) / kNT;
  const int top = nb - 1 - per * (int)threadIdx.x;
  uint32_t h[8];
  uint32_t local = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int b = top - j;
    h[j] = 0;
    if (j < per && b >= 0) h[j] = GLOBAL ? ld_acq(hist + b) : hist[b];
    local += h[j];
  }
  if (threadIdx.x == 0) { s_bin = -1; s_above = 0; }
  uint32_t total;
  const uint32_t excl = block_excl_scan(local, lds, total);
  if (excl < need && need <= excl + local) {
    uint32_t run = excl;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (j < per && run + h[j] >= need) { s_bin = top - j; s_above = run; break; }
      run += h[j];
    }
  }
  __syncthreads();
  above = s_above;
  const int bin = s_bin;
  __syncthreads();
  return bin;
}

// ---------------------------------------------------------------------------------------------
// Decoupled look-back.  Each chunk publishes one 64-bit word: flag (bits 63:62; 1 = aggregate of
// this chunk only, 2 = inclusive prefix) and two 31-bit counts.  Flag and counts travel in the
// same atomic word, so no fences are needed.  Every wait is bounded: on timeout the diagnostics
// word is flagged and the wait ends (the output is then wrong but the kernel still exits).
// ---------------------------------------------------------------------------------------------
__device__ __forceinline__ uint64_t lb_pack(uint32_t flag, uint32_t a, uint32_t b) {
  return ((uint64_t)flag << 62) | ((uint64_t)(a & 0x7FFFFFFFu) << 31) | (uint64_t)(b & 0x7FFFFFFFu);
}
__device__ __forceinline__ uint32_t lb_flag(uint64_t s) { return (uint32_t)(s >> 62); }
__device__ __forceinline__ uint32_t lb_a(uint64_t s) { return (uint32_t)(s >> 31) & 0x7FFFFFFFu; }
__device__ __forceinline__ uint32_t lb_b(uint64_t s) { return (uint32_t)s & 0x7FFFFFFFu; }

__device__ __forceinline__ void lb_publish(uint64_t* st, uint32_t flag, uint32_t a, uint32_t b) {
  __hip_atomic_store(st, lb_pack(flag, a, b), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Executed by one full wave.  Sums the counts of chunks c-1, c-2, ..., down to the nearest chunk
// that published an inclusive prefix (chunk `first` always does).
__device__ void lb_lookback(uint64_t* status, int c, int first, uint32_t& ea, uint32_t& eb,
                            uint32_t* diag) {
  const int lane = threadIdx.x & 63;
  uint32_t sa = 0, sb = 0;
  int base = c - 1;
  while (base >= first) {
    const int p = base - lane;
    const bool valid = p >= first;
    uint64_t s = 0;
    if (valid) {
      int spins = 0;
      s = __hip_atomic_load(status + p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      while (lb_flag(s) == 0) {
        __builtin_amdgcn_s_sleep(1);
        s = __hip_atomic_load(status + p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        if (++spins > kSpinLimit) {
          atomicOr(diag, kDiagSpinTimeout);
          s = lb_pack(2, 0, 0);
          break;
        }
      }
    }
    const uint64_t pm = __ballot(valid && lb_flag(s) == 2);
    const int stop = pm ? (__ffsll((unsigned long long)pm) - 1) : 63;
    const bool take = valid && lane <= stop;
    sa += wave_sum(take ? lb_a(s) : 0u);
    sb += wave_sum(take ? lb_b(s) : 0u);
    if (pm) break;
    base -= 64;
  }
  ea = sa;
  eb = sb;
}

}  // namespace efs
