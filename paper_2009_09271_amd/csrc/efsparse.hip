// efsparse host library: layouts, argument checking, workspace layout and kernel launches.
// The C ABI is declared in include/efsparse.h.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

#include "../../include/efsparse.h"
#include "ef_kernels.h"

using namespace efs;

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Packs int32 / uint64 host arrays into one blob with 256-byte aligned sub-arrays.
struct Blob {
  std::vector<uint8_t> bytes;
  size_t add(const void* src, size_t n) {
    const size_t at = align_up(bytes.size(), kAlign);
    bytes.resize(at + align_up(n, kAlign), 0);
    if (n) std::memcpy(bytes.data() + at, src, n);
    return at;
  }
  template <typename T> size_t add(const std::vector<T>& v) { return add(v.data(), v.size() * sizeof(T)); }
};

// Region table over a list space: region l is [base[l], base[l+1]); chunks of `tile` positions.
void chunk_cover(const std::vector<int32_t>& base, int64_t total, uint32_t tile, std::vector<int32_t>& sf,
                 std::vector<int32_t>& sl, std::vector<int32_t>& per_region) {
  const int L = (int)base.size() - 1;
  const int64_t n = (total + tile - 1) / tile;
  sf.assign(n, 0);
  sl.assign(n, 0);
  int l = 0;
  for (int64_t c = 0; c < n; ++c) {
    const int64_t lo = c * tile, hi = std::min<int64_t>(total, lo + tile);
    while (l + 1 < L && base[l + 1] <= lo) ++l;
    sf[c] = l;
    int m = l;
    while (m + 1 < L && base[m + 1] <= hi - 1) ++m;
    sl[c] = m;
  }
  per_region.assign(L, 0);
  for (int r = 0; r < L; ++r) {
    const int64_t first = base[r] / tile, last = (base[r + 1] - 1) / tile;
    per_region[r] = (int32_t)(last - first + 1);
  }
}

struct WsLayout {
  size_t diag = 0, tickets = 0, arrive = 0, res = 0, cnt = 0, hist = 0, st_stream = 0, st_emit = 0;
  size_t zero_bytes = 0, list_idx = 0, list_val = 0, list_key = 0, total = 0;
};

}  // namespace

struct ef_layout {
  int64_t d = 0;
  int32_t L = 0;
  double density = 0;
  int64_t block = 1;
  std::vector<int64_t> off64;
  double rk_sigma = 10.0, rk_extra = 64.0, rk_capmult = 1.0, tk_mult = 2.0, tk_extra = 65536.0;

  std::vector<int32_t> off, k, P, bl, nb, hb, nch, tk_base, tk_nlch, rk_base, rk_nlch;
  std::vector<int32_t> csf, csl, tk_lsf, tk_lsl, rk_lsf, rk_lsl;
  std::vector<uint64_t> tau;
  int64_t K = 0;
  int32_t nchunks = 0;
  int64_t tk_cap = 0, rk_cap = 0;
  int randk_levels = 1;  // list-level launches after the random-k candidate pass

  Blob blob;
  size_t o_off, o_k, o_P, o_bl, o_nb, o_hb, o_nch, o_tau, o_tkb, o_tkn, o_rkb, o_rkn, o_csf, o_csl, o_tlsf,
      o_tlsl, o_rlsf, o_rlsl;
  Tables T{};
  bool bound = false;

  void build();
  WsLayout ws_layout(int op) const;
};

void ef_layout::build() {
  const int32_t n = L;
  off.resize(n + 1);
  for (int i = 0; i <= n; ++i) off[i] = (int32_t)off64[i];
  k.resize(n);
  P.assign(n + 1, 0);
  bl.resize(n);
  nb.resize(n);
  hb.resize(n);
  tau.resize(n);
  tk_base.assign(n + 1, 0);
  rk_base.assign(n + 1, 0);
  randk_levels = 1;
  for (int l = 0; l < n; ++l) {
    const int64_t dl = off64[l + 1] - off64[l];
    // k per segment: round-half-up of density * d_l in double, clamped to [1, d_l]
    int64_t kl = (int64_t)std::floor(density * (double)dl + 0.5);
    kl = std::min<int64_t>(std::max<int64_t>(kl, 1), dl);
    k[l] = (int32_t)kl;
    P[l + 1] = P[l] + (int32_t)kl;
    const int64_t b = dl > block ? block : 1;
    bl[l] = (int32_t)b;
    nb[l] = (int32_t)((dl + b - 1) / b);
    // random-k candidate bound: expected candidates mu = k + sigma*sqrt(k) + extra
    const double mu = (double)kl + rk_sigma * std::sqrt((double)kl) + rk_extra;
    const double p = mu / (double)dl;
    uint64_t t;
    if (p >= 1.0) t = 1ull << 32;
    else t = (uint64_t)std::ceil(std::max(p, 0.0) * 4294967296.0);
    t = std::min<uint64_t>(std::max<uint64_t>(t, 2), 1ull << 32);
    tau[l] = t;
    int h = 0;
    while (h < 32 && ((t - 1) >> h) != 0) ++h;
    hb[l] = h;
    const int rest = h - std::min(11, h);
    randk_levels = std::max(randk_levels, (rest + 10) / 11);
    const double E = (double)dl * (double)t / 4294967296.0;
    const double capr = std::ceil(rk_capmult * (E + 10.0 * std::sqrt(E) + 64.0));
    const int64_t rc = std::min<int64_t>(std::max<int64_t>((int64_t)capr, 1), dl);
    rk_base[l + 1] = rk_base[l] + (int32_t)rc;
    const double ct = std::ceil(tk_mult * (double)kl + tk_extra);
    const int64_t tc = std::min<int64_t>(std::max<int64_t>((int64_t)ct, 1), dl);
    tk_base[l + 1] = tk_base[l] + (int32_t)tc;
  }
  K = P[n];
  tk_cap = tk_base[n];
  rk_cap = rk_base[n];
  nchunks = (int32_t)((d + kTile - 1) / kTile);
  chunk_cover(off, d, kTile, csf, csl, nch);
  chunk_cover(tk_base, tk_cap, kLTile, tk_lsf, tk_lsl, tk_nlch);
  chunk_cover(rk_base, rk_cap, kLTile, rk_lsf, rk_lsl, rk_nlch);

  blob = Blob();
  o_off = blob.add(off);
  o_k = blob.add(k);
  o_P = blob.add(P);
  o_bl = blob.add(bl);
  o_nb = blob.add(nb);
  o_hb = blob.add(hb);
  o_nch = blob.add(nch);
  o_tau = blob.add(tau);
  o_tkb = blob.add(tk_base);
  o_tkn = blob.add(tk_nlch);
  o_rkb = blob.add(rk_base);
  o_rkn = blob.add(rk_nlch);
  o_csf = blob.add(csf);
  o_csl = blob.add(csl);
  o_tlsf = blob.add(tk_lsf);
  o_tlsl = blob.add(tk_lsl);
  o_rlsf = blob.add(rk_lsf);
  o_rlsl = blob.add(rk_lsl);
  bound = false;
}

WsLayout ef_layout::ws_layout(int op) const {
  WsLayout w;
  const size_t Ls = (size_t)L;
  const size_t nl = op == EF_OP_TOPK ? tk_lsf.size() : rk_lsf.size();
  const size_t cap = op == EF_OP_TOPK ? (size_t)tk_cap : (size_t)rk_cap;
  size_t at = 0;
  w.diag = at;
  w.tickets = at + 4;
  at = 16;
  w.arrive = at;
  at += 3 * Ls * 4;
  w.res = at;
  at += Ls * kResWords * 4;
  w.cnt = at;
  at += Ls * 4;
  at = align_up(at, 16);
  w.hist = at;
  at += 3 * Ls * kHBins * 4;
  at = align_up(at, 16);
  w.st_stream = at;
  at += (size_t)nchunks * 8;
  w.st_emit = at;
  at += nl * 8;
  w.zero_bytes = align_up(at, 16);
  at = align_up(at, kAlign);
  w.list_idx = at;
  at = align_up(at + cap * 4, kAlign);
  w.list_val = at;
  at = align_up(at + cap * 4, kAlign);
  if (op == EF_OP_RANDK) {
    w.list_key = at;
    at = align_up(at + cap * 4, kAlign);
  }
  w.total = at;
  return w;
}

namespace {

WS make_ws(const WsLayout& l, void* base) {
  uint8_t* b = reinterpret_cast<uint8_t*>(base);
  WS w;
  w.diag = reinterpret_cast<uint32_t*>(b + l.diag);
  w.tickets = reinterpret_cast<uint32_t*>(b + l.tickets);
  w.arrive = reinterpret_cast<uint32_t*>(b + l.arrive);
  w.res = reinterpret_cast<uint32_t*>(b + l.res);
  w.cnt = reinterpret_cast<uint32_t*>(b + l.cnt);
  w.hist = reinterpret_cast<uint32_t*>(b + l.hist);
  w.st_stream = reinterpret_cast<uint64_t*>(b + l.st_stream);
  w.st_emit = reinterpret_cast<uint64_t*>(b + l.st_emit);
  w.list_idx = reinterpret_cast<uint32_t*>(b + l.list_idx);
  w.list_val = reinterpret_cast<float*>(b + l.list_val);
  w.list_key = l.list_key ? reinterpret_cast<uint32_t*>(b + l.list_key) : nullptr;
  return w;
}

hipStream_t S(void* s) { return reinterpret_cast<hipStream_t>(s); }

thread_local int g_last_hip_error = 0;

int hip_status(hipError_t e) {
  if (e == hipSuccess) return EF_OK;
  g_last_hip_error = (int)e;
  return EF_EHIP;
}

int launched() { return hip_status(hipGetLastError()); }

#define EF_TRY(x)              \
  do {                         \
    const int _rc = (x);       \
    if (_rc != EF_OK) return _rc; \
  } while (0)

int check_bound(const ef_layout* L) {
  if (!L || !L->bound) return EF_EINVAL;
  return EF_OK;
}

int check_g(const void* g, int g_dtype) {
  if (g_dtype == EF_F32) return g && aligned(g, 16) ? EF_OK : EF_EINVAL;
  if (g_dtype == EF_BF16) return g && aligned(g, 8) ? EF_OK : EF_EINVAL;
  return EF_EINVAL;
}

bool vec_ok(const void* p) { return p && aligned(p, 16); }
bool word_ok(const void* p) { return p && aligned(p, 4); }

int fill_zero(void* ws, size_t bytes, hipStream_t st) {
  const size_t words = bytes / 4;
  if (!words) return EF_OK;
  const size_t blocks = std::min<size_t>(1024, (words / 4 + kNT - 1) / kNT + 1);
  hipLaunchKernelGGL(k_fill_zero, dim3((unsigned)blocks), dim3(kNT), 0, st, reinterpret_cast<uint32_t*>(ws), words);
  return launched();
}

int check_ws(const ef_layout* L, int op, void* ws, size_t ws_bytes, WsLayout& wl) {
  wl = L->ws_layout(op);
  if (!ws || !aligned(ws, kAlign)) return EF_EINVAL;
  if (ws_bytes < wl.total) return EF_EWORKSPACE;
  return EF_OK;
}

// Top-k: level-0 histogram (fused with the accumulate when g != null), candidate list, last
// level, emission.
int run_topk(const ef_layout* L, const void* g, int g_dtype, const float* src, float* e_fused, uint32_t* idx,
             float* val, void* ws, size_t ws_bytes, void* stream) {
  WsLayout wl;
  EF_TRY(check_ws(L, EF_OP_TOPK, ws, ws_bytes, wl));
  hipStream_t st = S(stream);
  WS w = make_ws(wl, ws);
  const Tables& T = L->T;
  const dim3 grid((unsigned)L->nchunks), blk(kNT);
  const dim3 lgrid((unsigned)L->tk_lsf.size());
  EF_TRY(fill_zero(ws, wl.zero_bytes, st));
  if (g) {
    if (g_dtype == EF_F32)
      hipLaunchKernelGGL((k_topk_hist<0, true>), grid, blk, 0, st, T, g, src, e_fused, w);
    else
      hipLaunchKernelGGL((k_topk_hist<1, true>), grid, blk, 0, st, T, g, src, e_fused, w);
  } else {
    hipLaunchKernelGGL((k_topk_hist<0, false>), grid, blk, 0, st, T, nullptr, src, nullptr, w);
  }
  EF_TRY(launched());
  const float* acc = g ? e_fused : src;
  hipLaunchKernelGGL(k_topk_emit, grid, blk, 0, st, T, acc, w);
  EF_TRY(launched());
  hipLaunchKernelGGL(k_list_level<0>, lgrid, blk, 0, st, T, w, 2, acc, e_fused, idx, val, 0u, 0u, 0u);
  EF_TRY(launched());
  hipLaunchKernelGGL(k_list_emit<0>, lgrid, blk, 0, st, T, w, idx, val, e_fused);
  return launched();
}

int run_randk(const ef_layout* L, const void* g, int g_dtype, const float* src, float* e_fused, uint64_t seed,
              uint32_t step, uint32_t* idx, float* val, void* ws, size_t ws_bytes, void* stream) {
  WsLayout wl;
  EF_TRY(check_ws(L, EF_OP_RANDK, ws, ws_bytes, wl));
  hipStream_t st = S(stream);
  WS w = make_ws(wl, ws);
  const Tables& T = L->T;
  const dim3 grid((unsigned)L->nchunks), blk(kNT);
  const dim3 lgrid((unsigned)L->rk_lsf.size());
  const uint32_t s0 = (uint32_t)seed, s1 = (uint32_t)(seed >> 32);
  EF_TRY(fill_zero(ws, wl.zero_bytes, st));
  if (g) {
    if (g_dtype == EF_F32)
      hipLaunchKernelGGL((k_randk_stream<0, true>), grid, blk, 0, st, T, g, src, e_fused, s0, s1, step, w);
    else
      hipLaunchKernelGGL((k_randk_stream<1, true>), grid, blk, 0, st, T, g, src, e_fused, s0, s1, step, w);
  } else {
    hipLaunchKernelGGL((k_randk_stream<0, false>), grid, blk, 0, st, T, nullptr, src, nullptr, s0, s1, step, w);
  }
  EF_TRY(launched());
  const float* acc = g ? e_fused : src;
  for (int lev = 0; lev < L->randk_levels; ++lev) {
    hipLaunchKernelGGL(k_list_level<1>, lgrid, blk, 0, st, T, w, 1 + lev, acc, e_fused, idx, val, s0, s1, step);
    EF_TRY(launched());
  }
  hipLaunchKernelGGL(k_list_emit<1>, lgrid, blk, 0, st, T, w, idx, val, e_fused);
  return launched();
}

}  // namespace

// ============================================================================================
// C ABI
// ============================================================================================
extern "C" {

const char* ef_status_string(int status) {
  switch (status) {
    case EF_OK: return "EF_OK";
    case EF_EINVAL: return "EF_EINVAL: invalid argument";
    case EF_ERANGE: return "EF_ERANGE: size out of range";
    case EF_EWORKSPACE: return "EF_EWORKSPACE: workspace too small";
    case EF_EHIP: return "EF_EHIP: HIP runtime or launch error";
    default: return "unknown efsparse status";
  }
}

int ef_last_hip_error(void) { return g_last_hip_error; }

const char* ef_last_hip_error_string(void) {
  return g_last_hip_error ? hipGetErrorString((hipError_t)g_last_hip_error) : "no HIP error";
}

int ef_layout_create(int64_t d, const int64_t* seg_offsets, int32_t n_seg, double density, int64_t block,
                     ef_layout** out) {
  if (!out || !seg_offsets) return EF_EINVAL;
  if (d <= 0 || d >= (int64_t(1) << 31)) return EF_ERANGE;
  if (n_seg < 1 || n_seg >= (1 << 24)) return EF_ERANGE;
  if (!(density > 0.0 && density <= 1.0)) return EF_EINVAL;
  if (block < 1 || block > INT32_MAX) return EF_EINVAL;
  if (seg_offsets[0] != 0 || seg_offsets[n_seg] != d) return EF_EINVAL;
  for (int32_t i = 0; i < n_seg; ++i)
    if (seg_offsets[i + 1] <= seg_offsets[i]) return EF_EINVAL;
  ef_layout* L = new (std::nothrow) ef_layout();
  if (!L) return EF_EINVAL;
  L->d = d;
  L->L = n_seg;
  L->density = density;
  L->block = block;
  L->off64.assign(seg_offsets, seg_offsets + n_seg + 1);
  L->build();
  *out = L;
  return EF_OK;
}

int ef_layout_destroy(ef_layout* layout) {
  delete layout;
  return EF_OK;
}

int64_t ef_layout_total_k(const ef_layout* layout) { return layout ? layout->K : -1; }
int32_t ef_layout_num_segments(const ef_layout* layout) { return layout ? layout->L : -1; }

int ef_layout_segment_k(const ef_layout* layout, int64_t* k_out) {
  if (!layout || !k_out) return EF_EINVAL;
  for (int l = 0; l < layout->L; ++l) k_out[l] = layout->k[l];
  return EF_OK;
}

int ef_layout_tune(ef_layout* layout, int knob, double value) {
  if (!layout || !std::isfinite(value)) return EF_EINVAL;
  switch (knob) {
    case EF_TUNE_RANDK_SIGMA: layout->rk_sigma = value; break;
    case EF_TUNE_RANDK_EXTRA: layout->rk_extra = value; break;
    case EF_TUNE_TOPK_CAP_MULT: layout->tk_mult = value; break;
    case EF_TUNE_TOPK_CAP_EXTRA: layout->tk_extra = value; break;
    case EF_TUNE_RANDK_CAP_MULT: layout->rk_capmult = value; break;
    default: return EF_EINVAL;
  }
  layout->build();
  return EF_OK;
}

size_t ef_layout_device_bytes(const ef_layout* layout) { return layout ? layout->blob.bytes.size() : 0; }

int ef_layout_bind(ef_layout* L, void* dev, size_t bytes, void* stream) {
  if (!L || !dev || !aligned(dev, kAlign)) return EF_EINVAL;
  if (bytes < L->blob.bytes.size()) return EF_EWORKSPACE;
  hipStream_t st = S(stream);
  EF_TRY(hip_status(hipMemcpyAsync(dev, L->blob.bytes.data(), L->blob.bytes.size(), hipMemcpyHostToDevice, st)));
  EF_TRY(hip_status(hipStreamSynchronize(st)));
  uint8_t* b = reinterpret_cast<uint8_t*>(dev);
  Tables& T = L->T;
  T.seg_off = reinterpret_cast<const int32_t*>(b + L->o_off);
  T.seg_k = reinterpret_cast<const int32_t*>(b + L->o_k);
  T.seg_P = reinterpret_cast<const int32_t*>(b + L->o_P);
  T.seg_bl = reinterpret_cast<const int32_t*>(b + L->o_bl);
  T.seg_nb = reinterpret_cast<const int32_t*>(b + L->o_nb);
  T.seg_hb = reinterpret_cast<const int32_t*>(b + L->o_hb);
  T.seg_nchunks = reinterpret_cast<const int32_t*>(b + L->o_nch);
  T.seg_tau = reinterpret_cast<const uint64_t*>(b + L->o_tau);
  T.tk_base = reinterpret_cast<const int32_t*>(b + L->o_tkb);
  T.tk_nlch = reinterpret_cast<const int32_t*>(b + L->o_tkn);
  T.rk_base = reinterpret_cast<const int32_t*>(b + L->o_rkb);
  T.rk_nlch = reinterpret_cast<const int32_t*>(b + L->o_rkn);
  T.chunk_sf = reinterpret_cast<const int32_t*>(b + L->o_csf);
  T.chunk_sl = reinterpret_cast<const int32_t*>(b + L->o_csl);
  T.tk_lsf = reinterpret_cast<const int32_t*>(b + L->o_tlsf);
  T.tk_lsl = reinterpret_cast<const int32_t*>(b + L->o_tlsl);
  T.rk_lsf = reinterpret_cast<const int32_t*>(b + L->o_rlsf);
  T.rk_lsl = reinterpret_cast<const int32_t*>(b + L->o_rlsl);
  T.d = (int32_t)L->d;
  T.L = L->L;
  T.nchunks = L->nchunks;
  T.tk_nlchunks = (int32_t)L->tk_lsf.size();
  T.rk_nlchunks = (int32_t)L->rk_lsf.size();
  L->bound = true;
  return EF_OK;
}

size_t ef_workspace_bytes(const ef_layout* layout, int op, int32_t W) {
  if (!layout) return 0;
  switch (op) {
    case EF_OP_TOPK:
    case EF_OP_RANDK: return layout->ws_layout(op).total;
    case EF_OP_RANDBLOCK: return 0;
    case EF_OP_AGG_SPARSE:
      if (W < 1) return 0;
      return align_up((size_t)W * ((size_t)layout->nchunks + 1) * 4, kAlign);
    case EF_OP_AGG_BLOCK: return 0;
    default: return 0;
  }
}

size_t ef_workspace_diag_offset(const ef_layout* layout, int op) {
  if (!layout || (op != EF_OP_TOPK && op != EF_OP_RANDK)) return (size_t)-1;
  return layout->ws_layout(op).diag;
}

int ef_accumulate(const ef_layout* L, const void* g, int g_dtype, const float* e, float* acc, void* stream) {
  EF_TRY(check_bound(L));
  EF_TRY(check_g(g, g_dtype));
  if (!vec_ok(e) || !vec_ok(acc)) return EF_EINVAL;
  const dim3 grid((unsigned)L->nchunks), blk(kNT);
  if (g_dtype == EF_F32)
    hipLaunchKernelGGL(k_accumulate<0>, grid, blk, 0, S(stream), L->T.d, g, e, acc);
  else
    hipLaunchKernelGGL(k_accumulate<1>, grid, blk, 0, S(stream), L->T.d, g, e, acc);
  return launched();
}

int compress_topk(const ef_layout* L, const float* acc, uint32_t* idx, float* val, void* ws, size_t ws_bytes,
                  void* stream) {
  EF_TRY(check_bound(L));
  if (!vec_ok(acc) || !word_ok(idx) || !word_ok(val)) return EF_EINVAL;
  return run_topk(L, nullptr, EF_F32, acc, nullptr, idx, val, ws, ws_bytes, stream);
}

int ef_step_topk(const ef_layout* L, const void* g, int g_dtype, float* e, uint32_t* idx, float* val, void* ws,
                 size_t ws_bytes, void* stream) {
  EF_TRY(check_bound(L));
  EF_TRY(check_g(g, g_dtype));
  if (!vec_ok(e) || !word_ok(idx) || !word_ok(val)) return EF_EINVAL;
  return run_topk(L, g, g_dtype, e, e, idx, val, ws, ws_bytes, stream);
}

int compress_randk(const ef_layout* L, const float* acc, uint64_t seed, uint32_t step, uint32_t* idx, float* val,
                   void* ws, size_t ws_bytes, void* stream) {
  EF_TRY(check_bound(L));
  if (!vec_ok(acc) || !word_ok(idx) || !word_ok(val)) return EF_EINVAL;
  return run_randk(L, nullptr, EF_F32, acc, nullptr, seed, step, idx, val, ws, ws_bytes, stream);
}

int ef_step_randk(const ef_layout* L, const void* g, int g_dtype, float* e, uint64_t seed, uint32_t step,
                  uint32_t* idx, float* val, void* ws, size_t ws_bytes, void* stream) {
  EF_TRY(check_bound(L));
  EF_TRY(check_g(g, g_dtype));
  if (!vec_ok(e) || !word_ok(idx) || !word_ok(val)) return EF_EINVAL;
  return run_randk(L, g, g_dtype, e, e, seed, step, idx, val, ws, ws_bytes, stream);
}

int compress_randblock(const ef_layout* L, const float* acc, uint64_t seed, uint32_t step, uint32_t* start,
                       float* val, void* stream) {
  EF_TRY(check_bound(L));
  if (!vec_ok(acc) || !word_ok(start) || !word_ok(val)) return EF_EINVAL;
  const unsigned blocks = (unsigned)((L->K + kNT - 1) / kNT);
  hipLaunchKernelGGL(k_randblock_gather, dim3(blocks), dim3(kNT), 0, S(stream), L->T, (int32_t)L->K, acc,
                     (uint32_t)seed, (uint32_t)(seed >> 32), step, start, val);
  return launched();
}

int ef_step_randblock(const ef_layout* L, const void* g, int g_dtype, float* e, uint64_t seed, uint32_t step,
                      uint32_t* start, float* val, void* stream) {
  EF_TRY(check_bound(L));
  EF_TRY(check_g(g, g_dtype));
  if (!vec_ok(e) || !word_ok(start) || !word_ok(val)) return EF_EINVAL;
  const dim3 grid((unsigned)L->nchunks), blk(kNT);
  const uint32_t s0 = (uint32_t)seed, s1 = (uint32_t)(seed >> 32);
  if (g_dtype == EF_F32)
    hipLaunchKernelGGL(k_randblock_step<0>, grid, blk, 0, S(stream), L->T, g, e, s0, s1, step, start, val);
  else
    hipLaunchKernelGGL(k_randblock_step<1>, grid, blk, 0, S(stream), L->T, g, e, s0, s1, step, start, val);
  return launched();
}

int ef_update(const ef_layout* L, const float* acc, int msg_kind, const uint32_t* m, float* e, void* stream) {
  EF_TRY(check_bound(L));
  if (!vec_ok(acc) || !vec_ok(e) || !word_ok(m)) return EF_EINVAL;
  hipStream_t st = S(stream);
  const unsigned kblocks = (unsigned)((L->K + kNT - 1) / kNT);
  if (msg_kind == EF_MSG_SPARSE) {
    if (e != acc) {
      hipLaunchKernelGGL(k_copy, dim3((unsigned)L->nchunks), dim3(kNT), 0, st, L->T.d, acc, e);
      EF_TRY(launched());
    }
    hipLaunchKernelGGL(k_sparse_zero, dim3(kblocks), dim3(kNT), 0, st, L->T.d, (int32_t)L->K, m, e);
    return launched();
  }
  if (msg_kind == EF_MSG_BLOCK) {
    if (e == acc)
      hipLaunchKernelGGL(k_block_zero, dim3(kblocks), dim3(kNT), 0, st, L->T, (int32_t)L->K, m, e);
    else
      hipLaunchKernelGGL(k_block_update, dim3((unsigned)L->nchunks), dim3(kNT), 0, st, L->T, acc, m, e);
    return launched();
  }
  return EF_EINVAL;
}

int decompress_aggregate(const ef_layout* L, int msg_kind, int32_t W, const uint32_t* m, const float* val,
                         int average, float* out, void* ws, size_t ws_bytes, void* stream) {
  EF_TRY(check_bound(L));
  if (W < 1 || W > 65536) return EF_ERANGE;
  if (!word_ok(m) || !word_ok(val) || !vec_ok(out)) return EF_EINVAL;
  hipStream_t st = S(stream);
  const dim3 grid((unsigned)L->nchunks), blk(kNT);
  if (msg_kind == EF_MSG_SPARSE) {
    const size_t need = ef_workspace_bytes(L, EF_OP_AGG_SPARSE, W);
    if (!ws || !aligned(ws, kAlign)) return EF_EINVAL;
    if (ws_bytes < need) return EF_EWORKSPACE;
    const size_t entries = (size_t)W * (size_t)L->K;
    const size_t blocks = (entries + kNT - 1) / kNT;
    if (blocks > 0x7FFFFFFFu) return EF_ERANGE;
    uint32_t* ts = reinterpret_cast<uint32_t*>(ws);
    hipLaunchKernelGGL(k_agg_ranges, dim3((unsigned)blocks), blk, 0, st, L->T.d, W, (int32_t)L->K,
                       L->nchunks, m, ts);
    EF_TRY(launched());
    hipLaunchKernelGGL(k_agg_sparse, grid, blk, 0, st, L->T.d, W, (int32_t)L->K, L->nchunks, m, val, ts,
                       average, out);
    return launched();
  }
  if (msg_kind == EF_MSG_BLOCK) {
    hipLaunchKernelGGL(k_agg_block, grid, blk, 0, st, L->T, W, (int32_t)L->K, m, val, average, out);
    return launched();
  }
  return EF_EINVAL;
}

}  // extern "C"
