// efsparse host library: layouts, argument checking, workspace layout and kernel launches.
// The C ABI is declared in include/efsparse.h.

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/efsparse.h"
#include "ef_kernels.h"

using namespace efs;

// Scratch of decompress_aggregate_noalloc, for callers that cannot allocate device memory: the
// sparse aggregate's tile-range table.  Every device the library runs on holds its own copy until
// the process ends.  In host code this name only stands in for the device array: kernels and copies
// take the device address resolved by scratch_on(), never the name itself.
constexpr size_t kNoAllocScratch = (size_t)16 << 20;
static __device__ __align__(256) uint8_t scratch[kNoAllocScratch];

namespace {

constexpr size_t kAlign = 256;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
int32_t agg_tiles(int64_t d) { return (int32_t)((d + kAggTile - 1) / kAggTile); }
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

struct WsLayout {
  size_t diag = 0, res = 0, hist = 0, samp = 0, counts = 0, rcnt = 0, roff = 0, rtie = 0, lcnt = 0, coff = 0, pcnt = 0,
         cand_idx = 0, cand_val = 0, cand_key = 0, list_idx = 0, list_key = 0, total = 0;
  uint32_t S = 0, capB = 0;
};

}  // namespace

struct ef_layout {
  int64_t d = 0;
  int32_t L = 0;
  double density = 0;
  int64_t block = 1;
  std::vector<int64_t> off64;
  double rk_sigma = 6.0, rk_extra = 32.0, tk_sigma = 6.0, tk_extra = 8.0, tk_retry = 1.0, pool = 1.0;

  std::vector<int32_t> off, k, P, bl, nb, srank, urank, cbase, ro, csf, csl, rseg, runseg;
  std::vector<uint32_t> btile;  // block aggregate, multi-segment: (data tile, segment) pairs
  std::vector<uint32_t> rrec;   // multi-segment: per row (segment, its offset and end, tile base)
  std::vector<uint64_t> tau;
  std::vector<uint32_t> ulo;
  std::vector<uint64_t> lbase;      // per segment: list region
  std::vector<uint32_t> lq;         // entries per sub-list
  std::vector<uint32_t> zc;         // top-k, per segment: the fused pass stores +0 at the candidates
  std::vector<uint32_t> soff[2];    // per op (0 top-k, 1 random-k), per row: static slot start
  uint32_t S[2] = {64, 64};         // per op, one segment: static slot entries per row (at most)
  const uint32_t* dsoff[2] = {nullptr, nullptr};  // soff in the bound device tables
  uint64_t pB[2] = {0, 0}, lists = 0;  // overflow pool entries per op (0 top-k, 1 random-k), list entries
  int64_t K = 0;
  int32_t nchunks = 0, nrows = 0, nruns = 0;
  bool all_exact = false;  // top-k: every segment fits the sample, so the threshold is exact
  bool big = false;        // some k_l is large: row winners are counted by many workgroups
  bool rk_direct = false;  // random-k: every segment's rows and expected window fit k_select's LDS
  uint32_t rk_emit_rw = 16;  // random-k emission: rows per wavefront
  bool any_zc = false;       // some top-k segment stores +0 at its candidates in the fused pass

  Blob blob;
  size_t o_off, o_k, o_P, o_bl, o_nb, o_srank, o_urank, o_cbase, o_ro, o_tau, o_ulo, o_csf, o_csl, o_rseg, o_runseg,
      o_btile, o_rrec, o_lbase, o_lq, o_soff[2], o_zc;
  Tables T{};
  bool bound = false;
  bool valid = false;  // build() completed (host memory for the tables was available)

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
  srank.resize(n);
  urank.resize(n);
  tau.resize(n);
  ulo.resize(n);
  cbase.assign(n + 1, 0);
  ro.assign(n + 1, 0);
  all_exact = true;
  // top-k threshold sample: segments of more than kExactMax elements share the layout's samples in
  // proportion to their sizes (at least kSampleMinRuns runs each): kSampleTotal of them, or
  // kSampleCap at a density of 0.5 % or more when kSampleTotal would leave more than 10^6
  // candidates beyond the k_l (the margins of the sampled segments with 64 or more expected sampled
  // keys above their threshold, in elements).  A larger sample narrows the margin, and at such
  // densities every candidate beyond k_l is a loser whose value the emission writes back into e,
  // one scattered word each (1e9 elements: step 2.86 -> 2.67 ms at 1 %, 4.21 -> 3.93 ms at 10 %;
  // BERT flat at 10 %: 526 -> 510 us; where the margin holds few candidates, the longer sample
  // phase costs more than it saves).
  double dbig = 0.0;
  for (int l = 0; l < n; ++l)
    if (off64[l + 1] - off64[l] > kExactMax) dbig += (double)(off64[l + 1] - off64[l]);
  double excess = 0.0;
  for (int l = 0; l < n; ++l) {
    const double dl = (double)(off64[l + 1] - off64[l]);
    if (dl <= kExactMax) continue;
    const double nsl = (double)kSampleTotal * dl / dbig, mus = nsl * density;
    // (segments with few sampled keys above the threshold: the constant part of the margin
    // dominates there, and the excess candidates of a layer-wise layout are mostly not losers
    // written back: BERT per layer at 1 %, 384 -> 403 us with the larger sample)
    if (mus >= 64.0) excess += (tk_sigma * std::sqrt(mus) + tk_extra) * dl / nsl;
  }
  // Multi-segment layouts: the candidates beyond k_l expected under the base sample, with each
  // segment's own share (at least kSampleMinRuns runs).  Where they number over 4 million, four
  // times the larger sample: BERT per layer (4.9 and 6.6 million at 5 and 10 %) 489 -> 453 us and
  // 600 -> 576 us per step; with fewer the longer sample phase cost more than it saved (ResNet-18
  // per layer at 10 %, 0.5 million: 95 -> 113 us; BERT per layer at 1 %, 2.6 million, with the
  // larger sample alone: 384 -> 403 us).
  double lexcess = 0.0;
  for (int l = 0; l < n && n > 1; ++l) {
    const double dl = (double)(off64[l + 1] - off64[l]);
    if (dl <= kExactMax) continue;
    const double kl = std::min(std::max(std::floor(density * dl + 0.5), 1.0), dl);
    const double runs = std::min(std::max(std::ceil((double)kSampleTotal * dl / dbig / kSampleRun), (double)kSampleMinRuns),
                                 std::min((double)(kSampleCap / kSampleRun), std::floor(dl / kSampleRun)));
    const double ns = runs * kSampleRun, mus = ns * kl / dl;
    lexcess += std::min(std::ceil(mus + tk_sigma * std::sqrt(mus) + tk_extra), ns) * dl / ns - kl;
  }
  double sample_total = density >= 0.005 && excess > 1e6 ? (double)kSampleCap : (double)kSampleTotal;
  if (density >= 0.005 && lexcess > 4e6) sample_total = 4.0 * kSampleCap;
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
    // top-k sample runs: the whole segment when it fits the sample, else its share of the samples
    int64_t runs = (dl + kSampleRun - 1) / kSampleRun;
    if (dl > kExactMax) {
      const double want = std::ceil(sample_total * (double)dl / dbig / kSampleRun);
      runs = (int64_t)std::min<double>(std::max<double>(want, kSampleMinRuns), kSampleCap / kSampleRun);
      runs = std::min<int64_t>(runs, dl / kSampleRun);  // strata of one element or more
    }
    const double ns = (double)(runs * kSampleRun);
    // top-k: rank of the candidate threshold inside the segment's sample of ns keys, so that the
    // expected sample count above the true threshold plus tk_sigma standard deviations is covered
    const double mus = ns * (double)kl / (double)dl;
    const double rs = std::ceil(mus + tk_sigma * std::sqrt(mus) + tk_extra);
    srank[l] = (int32_t)std::min<double>(std::max<double>(rs, 1.0), ns);
    const double ru = std::floor(mus - tk_sigma * std::sqrt(mus));
    urank[l] = (int32_t)std::min<double>(std::max<double>(ru, 1.0), ns);
    // random-k: keys below tau are candidates; expected count k + sigma * sqrt(k) + extra
    const double mu = (double)kl + rk_sigma * std::sqrt((double)kl) + rk_extra;
    const double p = mu / (double)dl;
    uint64_t t;
    if (p >= 1.0) t = 1ull << 32;
    else t = (uint64_t)std::ceil(std::max(p, 0.0) * 4294967296.0);
    tau[l] = std::min<uint64_t>(std::max<uint64_t>(t, 1), 1ull << 32);
    // keys below ulo are expected k - sigma * sqrt(k) - extra times: all winners unless more than k
    const double mlo = (double)kl - rk_sigma * std::sqrt((double)kl) - rk_extra;
    const double plo = mlo / (double)dl;
    uint64_t u = 0;
    if (plo >= 1.0) u = tau[l];
    else if (plo > 0.0) u = (uint64_t)std::floor(plo * 4294967296.0);
    u = std::min<uint64_t>(u, tau[l]);
    ulo[l] = (uint32_t)std::min<uint64_t>(u, 0xFFFFFFFFull);
    // rows: one per data tile the segment touches
    const int64_t c0 = off64[l] / kTile, c1 = (off64[l + 1] - 1) / kTile;
    cbase[l + 1] = cbase[l] + (int32_t)(c1 - c0 + 1);
    ro[l + 1] = ro[l] + (int32_t)runs;
    if (dl > kExactMax) all_exact = false;
  }
  K = P[n];
  // many-workgroup row counting: a very large k_l, or a segment with more rows than k_select's
  // workgroup scans quickly (one workgroup walking 244,141 rows took 0.5-0.9 ms at 1e9 elements)
  big = *std::max_element(k.begin(), k.end()) >= kBigK;
  for (int l = 0; l < n && !big; ++l)
    if (cbase[l + 1] - cbase[l] > kBigRows) big = true;
  // random-k without k_collect: every row of a segment is held by a k_select thread and the
  // whole window [ulo, tau) fits k_select's LDS list (a window or a row list that overflows at
  // run time takes the exact path)
  rk_direct = !big;
  for (int l = 0; l < n && rk_direct; ++l) {
    const double dl = (double)(off64[l + 1] - off64[l]);
    const double wm = (double)(tau[l] - ulo[l]) / 4294967296.0 * dl;
    if (cbase[l + 1] - cbase[l] > (int32_t)(kSelNT * kSelPer) || wm + 8.0 * std::sqrt(wm) + 16.0 > (double)kListLds)
      rk_direct = false;
  }
  nrows = cbase[n];
  nruns = ro[n];
  // Candidate pools.  Each row keeps up to S_l candidates in a static slot (S_l: the expected
  // candidates of one of segment l's rows, plus a margin); a row with more reserves its entries in
  // the overflow pool.  The pool is sized by the candidate bound of each segment,
  // plus slack for the whole layout: top-k: the winners (exact segments) or the expected count
  // above the sampled threshold, twice, plus eight k_l for a retry (which aims at 4 k_l + 256
  // candidates); random-k: the binomial bound.  A row that does not fit sends its segment to the
  // exact path (same result, slower).
  {
    uint64_t bt = 0, br = 0, lsum = 0;
    std::vector<uint32_t> slot[2];  // per op, per segment: static slot entries per row
    double musum = 0.0;             // random-k: expected candidates of the whole layout
    slot[0].assign(n, 64);
    slot[1].assign(n, 64);
    lbase.assign(n, 0);
    lq.assign(n, 0);
    zc.assign(n, 0);
    for (int l = 0; l < n; ++l) {
      const double dl = (double)(off64[l + 1] - off64[l]), kl = (double)k[l];
      double et;
      if (dl <= kExactMax) {
        et = kl;
      } else {
        const double ns = (double)((ro[l + 1] - ro[l]) * kSampleRun);
        et = (double)srank[l] * dl / ns;
      }
      const uint64_t ct = dl <= kExactMax ? (uint64_t)kl : (uint64_t)std::min(dl, std::ceil(2.0 * et + 8.0 * kl + 256.0));
      // top-k residual: +0 stored at the candidates by the pass (their losers restored by the
      // emission) on dense sampled segments (k_l >= 0.5 % of d_l) whose candidates are not many
      // more than the winners (under 1.8 k_l expected), else +0 stored at the winners by the
      // emission; single words written into evicted lines cost a line read and a line write
      // each, so whichever set is smaller is written.  On sparse or small segments the winners
      // are few either way, and a layout with no such segment keeps the pass without the test
      // (ResNet-50 per layer, 57.6 against 61.9 us); segments sampled whole are left out for that
      // reason: their few winners did not pay for the test over the whole layout (ResNet-50 per
      // layer at 1 %, whose 4096-element layers qualified: 114.1 -> 110.7 us per step)
      zc[l] = dl > kExactMax && kl >= 0.005 * dl && et <= 1.8 * kl ? 1u : 0u;
      const double mu = (double)tau[l] / 4294967296.0 * dl;
      const uint64_t cr = (uint64_t)std::min(dl, std::ceil(mu + 8.0 * std::sqrt(mu) + 64.0));
      // slots: mu + 4 sqrt(mu) + 32 for top-k's mean mu per row (its candidates above the sampled
      // threshold, or the winners), mu + 8 sqrt(mu) + 32 for random-k's binomial count; multiples of
      // 32 entries, at most a tile
      const double nrl = (double)(cbase[l + 1] - cbase[l]);
      auto round_slot = [](double x) {
        return (uint32_t)std::min<double>(kTile, std::max(32.0, std::ceil(x / 32.0) * 32.0));
      };
      const double mt = (dl <= kExactMax ? kl : std::min(dl, et)) / nrl;
      const double mr = (double)tau[l] / 4294967296.0 * std::min(dl, (double)kTile);
      slot[0][l] = round_slot(mt + 4.0 * std::sqrt(mt) + 32.0);
      slot[1][l] = round_slot(mr + 8.0 * std::sqrt(mr) + 32.0);
      musum += mu;
      bt += ct;
      br += cr;
      // lists: sub-list c takes the entries of the segment's rows c, c + 16, ...; each of the
      // min(16, rows) sub-lists in use holds the segment's bound (up to 16 rows: one row each, at
      // most a tile) or an eighth of it, at most the elements of its rows; a sub-list that
      // overflows sends the segment to the exact path
      // (scaled by the pool knob)
      const uint64_t bl = std::max(ct, cr), nr = (uint64_t)(cbase[l + 1] - cbase[l]);
      const uint64_t rows_cap = (nr + kSubLists - 1) / kSubLists * kTile;
      const uint64_t q0 = nr <= kSubLists ? std::min<uint64_t>(bl, kTile) : std::min<uint64_t>(bl, (bl + 7) / 8 + 64);
      const uint64_t q = std::min<uint64_t>(rows_cap, (uint64_t)std::ceil((double)q0 * pool));
      lbase[l] = lsum;
      lq[l] = (uint32_t)q;
      lsum += q * std::min<uint64_t>(nr, kSubLists);
    }
    for (int o = 0; o < 2; ++o) {
      S[o] = slot[o][0];
      soff[o].assign(nrows + 1, 0);
      for (int l = 0; l < n; ++l)
        for (int32_t r = cbase[l]; r < cbase[l + 1]; ++r) {
          const int64_t tb = (off64[l] / kTile + (r - cbase[l])) * kTile;
          const int64_t len = std::min<int64_t>(off64[l + 1], tb + kTile) - std::max<int64_t>(off64[l], tb);
          soff[o][r + 1] = soff[o][r] + (uint32_t)std::min<int64_t>(slot[o][l], len);
        }
    }
    // random-k emission: about 96 candidates per wavefront on average (16 rows of a few at low
    // density; at 1 % a wavefront of 16 rows walked ~650 candidates in turn)
    rk_emit_rw = 16;
    while (rk_emit_rw > 1 && (double)rk_emit_rw * musum / (double)std::max(nrows, 1) > 96.0) rk_emit_rw /= 2;
    pB[0] = (uint64_t)std::ceil((double)(bt + 49152 + kPools * 4096) * pool / kPools) * kPools;
    pB[1] = (uint64_t)std::ceil((double)(br + 49152 + kPools * 4096) * pool / kPools) * kPools;
    lists = lsum;
    any_zc = std::find(zc.begin(), zc.end(), 1u) != zc.end();
  }
  rseg.resize(nrows);
  for (int l = 0; l < n; ++l)
    for (int32_t r = cbase[l]; r < cbase[l + 1]; ++r) rseg[r] = l;
  rrec.clear();
  if (n > 1) {
    for (int l = 0; l < n; ++l)
      for (int32_t r = cbase[l]; r < cbase[l + 1]; ++r) {
        const uint32_t rec[4] = {(uint32_t)l, (uint32_t)off64[l], (uint32_t)off64[l + 1],
                                 (uint32_t)((off64[l] / kTile + (r - cbase[l])) * kTile)};
        rrec.insert(rrec.end(), rec, rec + 4);
      }
  }
  runseg.resize(nruns);
  for (int l = 0; l < n; ++l)
    for (int32_t r = ro[l]; r < ro[l + 1]; ++r) runseg[r] = l;
  nchunks = (int32_t)((d + kTile - 1) / kTile);
  csf.assign(nchunks, 0);
  csl.assign(nchunks, 0);
  int l = 0;
  for (int32_t c = 0; c < nchunks; ++c) {
    const int64_t lo = (int64_t)c * kTile, hi = std::min<int64_t>(d, lo + kTile);
    while (l + 1 < n && off64[l + 1] <= lo) ++l;
    csf[c] = l;
    int m = l;
    while (m + 1 < n && off64[m + 1] <= hi - 1) ++m;
    csl[c] = m;
  }

  // block aggregate over several segments: every (1024-element data tile, segment) pair with an
  // element in common, segment by segment, with the segment's offset, size, k and message offset
  // (eight words: the kernel loads a pair's record in one round trip)
  btile.clear();
  if (n > 1) {
    for (int s = 0; s < n; ++s) {
      const int64_t t0 = off64[s] / kAggBT, t1 = (off64[s + 1] - 1) / kAggBT;
      for (int64_t t = t0; t <= t1; ++t) {
        const uint32_t rec[kBtWords] = {(uint32_t)t, (uint32_t)s, (uint32_t)off64[s],
                                        (uint32_t)(off64[s + 1] - off64[s]), (uint32_t)k[s], (uint32_t)P[s], 0u, 0u};
        btile.insert(btile.end(), rec, rec + kBtWords);
      }
    }
  }

  blob = Blob();
  o_off = blob.add(off);
  o_k = blob.add(k);
  o_P = blob.add(P);
  o_bl = blob.add(bl);
  o_nb = blob.add(nb);
  o_srank = blob.add(srank);
  o_urank = blob.add(urank);
  o_cbase = blob.add(cbase);
  o_ro = blob.add(ro);
  o_tau = blob.add(tau);
  o_ulo = blob.add(ulo);
  o_csf = blob.add(csf);
  o_csl = blob.add(csl);
  o_rseg = blob.add(rseg);
  o_runseg = blob.add(runseg);
  o_btile = blob.add(btile);
  o_rrec = blob.add(rrec);
  o_lbase = blob.add(lbase);
  o_zc = blob.add(zc);
  o_lq = blob.add(lq);
  o_soff[0] = blob.add(soff[0]);
  o_soff[1] = blob.add(soff[1]);
  bound = false;
}

WsLayout ef_layout::ws_layout(int op) const {
  WsLayout w;
  size_t at = 0;
  auto take = [&](size_t bytes) {
    const size_t a = at;
    at = align_up(at + bytes, kAlign);
    return a;
  };
  const size_t rows = (size_t)nrows;
  const int o = op == EF_OP_TOPK ? 0 : 1;
  w.S = soff[o][rows];  // the static slots' total: the overflow pool starts there
  // at most every element once more (a pass whose rows all overflow their static slots); entry
  // positions are 32-bit: the pool ends below 2^32
  const uint64_t every = ((uint64_t)d + kPools * 4096 + kPools - 1) / kPools * kPools;
  w.capB = (uint32_t)std::min<uint64_t>({pB[o], every, (0xFFFFFFFEull - w.S) / kPools * kPools});
  const size_t slots = (size_t)w.S + w.capB;  // candidate pool entries
  // the segments' sub-lists; random-k's direct lists instead: a (key', index) pair for each pool
  // entry, in the list_idx memory
  const bool pairs = o == 1 && rk_direct;
  w.diag = take(16);
  w.res = take((size_t)L * kResWords * 4);
  w.hist = take((size_t)L * kHCopies * kHBins * 4);
  w.samp = op == EF_OP_TOPK ? take((size_t)nruns * kSampleRun * 4) : 0;
  w.counts = take(rows * 4);
  w.rcnt = take(rows * 4);
  w.roff = take(rows * 4);
  w.rtie = take(rows * 4);
  w.lcnt = take((size_t)L * kSubLists * kLineWords * 4);
  w.coff = take(rows * 4);
  w.pcnt = take((size_t)kPools * kLineWords * 4);
  w.cand_idx = take(slots * 4);
  w.cand_val = take(slots * 4);
  w.cand_key = take(slots * 4);
  w.list_idx = take(pairs ? slots * 8 : (size_t)lists * 4);
  w.list_key = take(pairs ? 0 : (size_t)lists * 4);
  w.total = at;
  return w;
}

namespace {

WSel make_ws(const WsLayout& l, void* base) {
  uint8_t* b = reinterpret_cast<uint8_t*>(base);
  WSel w;
  w.diag = reinterpret_cast<uint32_t*>(b + l.diag);
  w.res = reinterpret_cast<uint32_t*>(b + l.res);
  w.hist = reinterpret_cast<uint32_t*>(b + l.hist);
  w.samp = reinterpret_cast<uint32_t*>(b + l.samp);
  w.counts = reinterpret_cast<uint32_t*>(b + l.counts);
  w.rcnt = reinterpret_cast<uint32_t*>(b + l.rcnt);
  w.roff = reinterpret_cast<uint32_t*>(b + l.roff);
  w.rtie = reinterpret_cast<uint32_t*>(b + l.rtie);
  w.lcnt = reinterpret_cast<uint32_t*>(b + l.lcnt);
  w.coff = reinterpret_cast<uint32_t*>(b + l.coff);
  w.pcnt = reinterpret_cast<uint32_t*>(b + l.pcnt);
  w.pool0 = l.S;
  w.capB = l.capB;
  w.cand_idx = reinterpret_cast<uint32_t*>(b + l.cand_idx);
  w.cand_val = reinterpret_cast<float*>(b + l.cand_val);
  w.cand_key = reinterpret_cast<uint32_t*>(b + l.cand_key);
  w.list_idx = reinterpret_cast<uint32_t*>(b + l.list_idx);
  w.list_key = reinterpret_cast<uint32_t*>(b + l.list_key);
  w.pairs = reinterpret_cast<uint2*>(b + l.list_idx);
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

// ---- optional per-kernel timing: HIP events recorded around each launch on its stream ----
struct TimingRec {
  const char* name;
  hipEvent_t a, b;
};
struct TimingAgg {
  std::string name;
  double ms;
  int64_t n;
};
std::mutex g_tm;
std::atomic<bool> g_timing{false};  // read on every launch without the lock
std::vector<TimingRec> g_pending;
std::vector<hipEvent_t> g_pool;
std::vector<TimingAgg> g_totals;

hipEvent_t pool_event() {
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// While timing is on, a launch gets a start and a stop event that the runtime ties to the kernel's
// own dispatch (hipExtLaunchKernelGGL), so the elapsed time is the kernel's execution alone.
bool timing_slot(const char* name, hipEvent_t* a, hipEvent_t* b) {
  if (!g_timing.load(std::memory_order_relaxed)) return false;
  std::lock_guard<std::mutex> lk(g_tm);
  TimingRec r{name, pool_event(), pool_event()};
  if (!r.a || !r.b) return false;
  try {
    g_pending.push_back(r);
  } catch (const std::bad_alloc&) {  // no room to record it: the launch goes untimed
    g_pool.push_back(r.a);
    g_pool.push_back(r.b);
    return false;
  }
  *a = r.a;
  *b = r.b;
  return true;
}

// Every launch goes through this macro: the kernel is named after its expression.
#define EF_LAUNCH(KERNEL, GRID, BLOCK, SHM, ST, ...)                                   \
  do {                                                                                 \
    hipEvent_t _ea = nullptr, _eb = nullptr;                                           \
    if (timing_slot(#KERNEL, &_ea, &_eb))                                              \
      hipExtLaunchKernelGGL(KERNEL, GRID, BLOCK, SHM, ST, _ea, _eb, 0u, __VA_ARGS__); \
    else                                                                               \
      hipLaunchKernelGGL(KERNEL, GRID, BLOCK, SHM, ST, __VA_ARGS__);                  \
  } while (0)

#define EF_TRY(x)              \
  do {                         \
    const int _rc = (x);       \
    if (_rc != EF_OK) return _rc; \
  } while (0)

int check_bound(const ef_layout* L) {
  if (!L || !L->valid || !L->bound) return EF_EINVAL;
  return EF_OK;
}

int check_g(const void* g, int g_dtype) {
  if (g_dtype == EF_F32) return g && aligned(g, 16) ? EF_OK : EF_EINVAL;
  if (g_dtype == EF_BF16) return g && aligned(g, 8) ? EF_OK : EF_EINVAL;
  return EF_EINVAL;
}

bool vec_ok(const void* p) { return p && aligned(p, 16); }
bool word_ok(const void* p) { return p && aligned(p, 4); }

int check_ws(const ef_layout* L, int op, void* ws, size_t ws_bytes, WsLayout& wl) {
  wl = L->ws_layout(op);
  if (!ws || !aligned(ws, kAlign)) return EF_EINVAL;
  if (ws_bytes < wl.total) return EF_EWORKSPACE;
  return EF_OK;
}

// The steps of W workers (one for the single-worker entry points): each worker's gradient and
// residual by pointer (host tables), messages of K entries and workspaces ws_stride bytes apart.
struct Steps {
  int32_t W = 1;
  const void* const* g = nullptr;  // [W]; null table: compress only (acc = src)
  int g_dtype = EF_F32;
  const float* const* src = nullptr;  // [W]: acc (compress) or e (fused step)
  float* const* e = nullptr;          // [W] or null table (compress)
  uint32_t* idx = nullptr;
  float* val = nullptr;
  uint8_t* ws = nullptr;
  size_t ws_bytes = 0;  // per worker
  size_t ws_stride = 0;
  const uint64_t* seeds = nullptr;  // random-k, host array [W]
  uint32_t step = 0;
};

// Top-k (KIND 0): sample -> candidate rule -> fused accumulate + candidates -> bin of the k-th ->
// collect -> exact threshold and row offsets -> emission.
// Random-k (KIND 1): fused accumulate + Philox candidates -> collect (certain winners counted, the
// window [ulo, tau) listed; on direct layouts by the streaming pass itself) -> exact threshold and
// row offsets -> emission.
// Each phase runs for all W workers before the next: the streaming passes one launch per worker,
// every other kernel once per kBatchMax workers (the worker is the grid's second dimension), so
// the short latency-bound selection kernels are paid once for the batch.
constexpr int kWideBatch = 8;  // batches of at least this many workers take the batch forms
constexpr uint64_t kWideRows = 131072;  // ... and so do sparse calls with this many rows in all

template <int KIND>
int run_select(const ef_layout* L, const Steps& P, unsigned phases, void* stream) {
  WsLayout wl;
  EF_TRY(check_ws(L, KIND == 0 ? EF_OP_TOPK : EF_OP_RANDK, P.ws, P.ws_bytes, wl));
  hipStream_t st = S(stream);
  const Tables& T = L->T;
  const uint64_t K = (uint64_t)L->K;
  const dim3 blk(kNT), sblk(kSelNT), pblk(kSampleRun);
  auto g_at = [&](int w) -> const void* { return P.g ? P.g[w] : nullptr; };
  auto e_at = [&](int w) -> float* { return P.e ? P.e[w] : nullptr; };
  auto ws_of = [&](int w) {
    WSel s = make_ws(wl, P.ws + (uint64_t)w * P.ws_stride);
    s.soff = L->dsoff[KIND];
    s.S = L->S[KIND];
    return s;
  };
  // the kernel-argument table of workers [c0, c0 + nw)
  auto batch_of = [&](int c0, int nw) {
    Batch b{};
    b.ws = P.ws_stride;
    b.msg = (uint32_t)K;
    for (int j = 0; j < nw; ++j) {
      b.g[j] = g_at(c0 + j);
      b.src[j] = P.src[c0 + j];
      b.e[j] = e_at(c0 + j);
      const uint64_t s = KIND == 1 && P.seeds ? P.seeds[c0 + j] : 0u;
      b.seed_lo[j] = (uint32_t)s;
      b.seed_hi[j] = (uint32_t)(s >> 32);
    }
    return b;
  };

  if (KIND == 0 && (phases & EF_PHASE_PREPARE)) {  // the sample and the candidate rule
    for (int c0 = 0; c0 < P.W; c0 += kBatchMax) {
      const unsigned nw = (unsigned)std::min(kBatchMax, P.W - c0);
      const WSel w = ws_of(c0);
      const Batch bt = batch_of(c0, (int)nw);
      const dim3 pgrid((unsigned)L->nruns, nw), sgrid((unsigned)L->L, nw);
      if (!P.g) EF_LAUNCH((k_sample_gather<0, false>), pgrid, pblk, 0, st, T, w, bt);
      else if (P.g_dtype == EF_F32) EF_LAUNCH((k_sample_gather<0, true>), pgrid, pblk, 0, st, T, w, bt);
      else EF_LAUNCH((k_sample_gather<1, true>), pgrid, pblk, 0, st, T, w, bt);
      EF_TRY(launched());
      EF_LAUNCH(k_sample_select, sgrid, sblk, 0, st, T, w, bt);
      EF_TRY(launched());
    }
  }
  if (phases & EF_PHASE_STREAM) {  // the streaming passes
    const dim3 rgrid((unsigned)L->nrows), rblk(kStrNT);
    for (int wk = 0; wk < P.W; ++wk) {
      const WSel w = ws_of(wk);
      const float* src = P.src[wk];
      const uint64_t seed = KIND == 1 && P.seeds ? P.seeds[wk] : 0u;
      const uint32_t s0 = (uint32_t)seed, s1 = (uint32_t)(seed >> 32), step = KIND == 1 ? P.step : 0u;
      if (!P.g)
        EF_LAUNCH((k_stream_sel<KIND, 0, false>), rgrid, rblk, 0, st, T, nullptr, src, nullptr, s0, s1, step, w);
      else if (KIND == 0 && L->any_zc && P.g_dtype == EF_F32)
        EF_LAUNCH((k_stream_sel<KIND, 0, true, true>), rgrid, rblk, 0, st, T, g_at(wk), src, e_at(wk), s0, s1, step, w);
      else if (KIND == 0 && L->any_zc)
        EF_LAUNCH((k_stream_sel<KIND, 1, true, true>), rgrid, rblk, 0, st, T, g_at(wk), src, e_at(wk), s0, s1, step, w);
      else if (P.g_dtype == EF_F32)
        EF_LAUNCH((k_stream_sel<KIND, 0, true>), rgrid, rblk, 0, st, T, g_at(wk), src, e_at(wk), s0, s1, step, w);
      else
        EF_LAUNCH((k_stream_sel<KIND, 1, true>), rgrid, rblk, 0, st, T, g_at(wk), src, e_at(wk), s0, s1, step, w);
      EF_TRY(launched());
    }
  }
  if (!(phases & EF_PHASE_FINISH)) return EF_OK;
  for (int c0 = 0; c0 < P.W; c0 += kBatchMax) {
    const unsigned nw = (unsigned)std::min(kBatchMax, P.W - c0);
    const WSel w = ws_of(c0);
    const Batch bt = batch_of(c0, (int)nw);
    const dim3 sgrid((unsigned)L->L, nw);
    // rows per wavefront of the collection and of the emission: top-k rows hold hundreds of
    // candidates, so one row per wavefront for one or a few workers (the most parallel form) and,
    // for a batch, two (collection) or four (emission) for fewer, fuller wavefronts (measured on
    // 16 workers: collection 23.7 us with two, 25.8 with four; emission the same with two or
    // four); random-k rows hold a few at low density, 16 per wavefront there, fewer as the density
    // grows (rk_emit_rw)
    // (one worker on a very large, sparse layout as well: 1e9 elements at 0.01-0.1 %, top-k
    // emission 79-87 -> 28-39 us; at 1-10 %, with hundreds of candidates a row, it was slower)
    const bool wide = nw >= kWideBatch ||
                      ((uint64_t)nw * L->nrows >= kWideRows && (uint64_t)L->K <= 16ull * L->nrows);
    const uint32_t emit_rw = KIND == 1 ? L->rk_emit_rw : wide ? 4u : 1u;
    const uint32_t emit_rows = (kNT / 64) * emit_rw;
    const dim3 egrid((unsigned)((L->nrows + emit_rows - 1) / emit_rows), nw);
    uint32_t* idx = P.idx + (uint64_t)c0 * K;
    float* val = P.val ? P.val + (uint64_t)c0 * K : nullptr;  // none: a selection prepared ahead
    if (KIND == 0 ? !L->all_exact : !L->rk_direct) {
      if (KIND == 0) {
        EF_LAUNCH(k_resolve, sgrid, sblk, 0, st, T, w, bt);
        EF_TRY(launched());
      }
      const uint32_t crows = (kNT / 64) * (wide ? 2u : 1u);  // rows per workgroup
      const dim3 cgrid((unsigned)((L->nrows + crows - 1) / crows), nw);
      if (wide) EF_LAUNCH((k_collect<KIND, 2>), cgrid, blk, 0, st, T, w, bt);
      else EF_LAUNCH((k_collect<KIND, 1>), cgrid, blk, 0, st, T, w, bt);
      EF_TRY(launched());
    }
    if (L->big) {
      EF_LAUNCH((k_select<KIND, true>), sgrid, sblk, 0, st, T, w, idx, val, P.step, bt);
      EF_TRY(launched());
      const dim3 cgrid1((unsigned)((L->nrows + kNT / 64 - 1) / (kNT / 64)), nw);  // a row per wavefront
      EF_LAUNCH(k_rowcount<KIND>, cgrid1, blk, 0, st, T, w, bt);
      EF_TRY(launched());
      EF_LAUNCH(k_rowscan, sgrid, sblk, 0, st, T, w, bt);
    } else {
      EF_LAUNCH((k_select<KIND, false>), sgrid, sblk, 0, st, T, w, idx, val, P.step, bt);
    }
    EF_TRY(launched());
    const int cz = KIND == 1 && P.e ? 1 : 0;  // random-k, fused: the candidates were stored as +0
    // (top-k rows with winning ties are emitted from acc)
    if (emit_rw == 16u) EF_LAUNCH((k_emit<16, KIND == 0>), egrid, blk, 0, st, T, w, idx, val, bt, cz);
    else if (emit_rw == 8u) EF_LAUNCH((k_emit<8, KIND == 0>), egrid, blk, 0, st, T, w, idx, val, bt, cz);
    else if (emit_rw == 4u) EF_LAUNCH((k_emit<4, KIND == 0>), egrid, blk, 0, st, T, w, idx, val, bt, cz);
    else if (emit_rw == 2u) EF_LAUNCH((k_emit<2, KIND == 0>), egrid, blk, 0, st, T, w, idx, val, bt, cz);
    else EF_LAUNCH((k_emit<1, KIND == 0>), egrid, blk, 0, st, T, w, idx, val, bt, cz);
    EF_TRY(launched());
  }
  return EF_OK;
}

// One worker's step (the single-worker entry points): pointer tables of one entry.
int run_one(int kind, const ef_layout* L, const void* g, int g_dtype, const float* src, float* e_fused, uint64_t seed,
            uint32_t step, uint32_t* idx, float* val, void* ws, size_t ws_bytes, void* stream, unsigned phases) {
  const void* gt[1] = {g};
  const float* st[1] = {src};
  float* et[1] = {e_fused};
  Steps P;
  P.g = g ? gt : nullptr;
  P.g_dtype = g_dtype;
  P.src = st;
  P.e = e_fused ? et : nullptr;
  P.idx = idx;
  P.val = val;
  P.ws = static_cast<uint8_t*>(ws);
  P.ws_bytes = ws_bytes;
  P.seeds = &seed;
  P.step = step;
  return kind == 0 ? run_select<0>(L, P, phases, stream) : run_select<1>(L, P, phases, stream);
}

int run_topk(const ef_layout* L, const void* g, int g_dtype, const float* src, float* e_fused, uint32_t* idx,
             float* val, void* ws, size_t ws_bytes, void* stream, unsigned phases = EF_PHASE_ALL) {
  return run_one(0, L, g, g_dtype, src, e_fused, 0u, 0u, idx, val, ws, ws_bytes, stream, phases);
}

int run_randk(const ef_layout* L, const void* g, int g_dtype, const float* src, float* e_fused, uint64_t seed,
              uint32_t step, uint32_t* idx, float* val, void* ws, size_t ws_bytes, void* stream,
              unsigned phases = EF_PHASE_ALL) {
  return run_one(1, L, g, g_dtype, src, e_fused, seed, step, idx, val, ws, ws_bytes, stream, phases);
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
    case EF_ENOMEM: return "EF_ENOMEM: out of host memory";
    default: return "unknown efsparse status";
  }
}

int ef_last_hip_error(void) { return g_last_hip_error; }

const char* ef_last_hip_error_string(void) {
  return g_last_hip_error ? hipGetErrorString((hipError_t)g_last_hip_error) : "no HIP error";
}

int ef_timing_enable(int enable) {
  std::lock_guard<std::mutex> lk(g_tm);
  g_timing.store(enable != 0);
  return EF_OK;
}

int ef_timing_collect(void) {
  std::lock_guard<std::mutex> lk(g_tm);
  int rc = EF_OK;
  for (const TimingRec& r : g_pending) {
    float ms = 0.f;
    if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) rc = EF_EHIP;
    TimingAgg* agg = nullptr;
    for (TimingAgg& t : g_totals)
      if (t.name == r.name) agg = &t;
    try {
      if (!agg) {
        g_totals.push_back(TimingAgg{r.name, 0.0, 0});
        agg = &g_totals.back();
      }
      g_pool.push_back(r.a);
      g_pool.push_back(r.b);
    } catch (const std::bad_alloc&) {
      rc = EF_ENOMEM;
    }
    if (agg) {
      agg->ms += ms;
      agg->n += 1;
    }
  }
  g_pending.clear();
  return rc;
}

int ef_timing_count(void) {
  std::lock_guard<std::mutex> lk(g_tm);
  return (int)g_totals.size();
}

int ef_timing_get(int i, const char** name, double* total_ms, int64_t* launches) {
  std::lock_guard<std::mutex> lk(g_tm);
  if (i < 0 || i >= (int)g_totals.size() || !name || !total_ms || !launches) return EF_EINVAL;
  *name = g_totals[i].name.c_str();
  *total_ms = g_totals[i].ms;
  *launches = g_totals[i].n;
  return EF_OK;
}

int ef_timing_reset(void) {
  std::lock_guard<std::mutex> lk(g_tm);
  g_totals.clear();
  return EF_OK;
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
  if (!L) return EF_ENOMEM;
  L->d = d;
  L->L = n_seg;
  L->density = density;
  L->block = block;
  // the tables are host vectors: an allocation failure ends here as a status, never as an
  // exception through the C ABI
  try {
    L->off64.assign(seg_offsets, seg_offsets + n_seg + 1);
    L->build();
  } catch (const std::bad_alloc&) {
    delete L;
    return EF_ENOMEM;
  }
  L->valid = true;
  *out = L;
  return EF_OK;
}

int ef_layout_destroy(ef_layout* layout) {
  delete layout;
  return EF_OK;
}

int64_t ef_layout_total_k(const ef_layout* layout) { return layout && layout->valid ? layout->K : -1; }
int32_t ef_layout_num_segments(const ef_layout* layout) { return layout ? layout->L : -1; }

int ef_layout_segment_k(const ef_layout* layout, int64_t* k_out) {
  if (!layout || !layout->valid || !k_out) return EF_EINVAL;
  for (int l = 0; l < layout->L; ++l) k_out[l] = layout->k[l];
  return EF_OK;
}

int ef_layout_tune(ef_layout* layout, int knob, double value) {
  if (!layout || !std::isfinite(value)) return EF_EINVAL;
  switch (knob) {
    case EF_TUNE_RANDK_SIGMA: layout->rk_sigma = value; break;
    case EF_TUNE_RANDK_EXTRA: layout->rk_extra = value; break;
    case EF_TUNE_TOPK_SIGMA: layout->tk_sigma = value; break;
    case EF_TUNE_TOPK_EXTRA: layout->tk_extra = value; break;
    case EF_TUNE_TOPK_RETRY: layout->tk_retry = value; break;
    case EF_TUNE_POOL:
      if (value < 0.0) return EF_EINVAL;
      layout->pool = value;
      break;
    default: return EF_EINVAL;
  }
  // a failed rebuild leaves the layout unusable (every later call on it returns EF_EINVAL)
  layout->valid = false;
  layout->bound = false;
  try {
    layout->build();
  } catch (const std::bad_alloc&) {
    return EF_ENOMEM;
  }
  layout->valid = true;
  return EF_OK;
}

size_t ef_layout_device_bytes(const ef_layout* layout) {
  return layout && layout->valid ? layout->blob.bytes.size() : 0;
}

int ef_layout_bind(ef_layout* L, void* dev, size_t bytes, void* stream) {
  if (!L || !L->valid || !dev || !aligned(dev, kAlign)) return EF_EINVAL;
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
  T.seg_srank = reinterpret_cast<const int32_t*>(b + L->o_srank);
  T.seg_urank = reinterpret_cast<const int32_t*>(b + L->o_urank);
  T.seg_cbase = reinterpret_cast<const int32_t*>(b + L->o_cbase);
  T.seg_ro = reinterpret_cast<const int32_t*>(b + L->o_ro);
  T.row_seg = reinterpret_cast<const int32_t*>(b + L->o_rseg);
  T.run_seg = reinterpret_cast<const int32_t*>(b + L->o_runseg);
  T.row_rec = reinterpret_cast<const uint32_t*>(b + L->o_rrec);
  T.seg_tau = reinterpret_cast<const uint64_t*>(b + L->o_tau);
  T.seg_ulo = reinterpret_cast<const uint32_t*>(b + L->o_ulo);
  T.seg_lbase = reinterpret_cast<const uint64_t*>(b + L->o_lbase);
  T.seg_lq = reinterpret_cast<const uint32_t*>(b + L->o_lq);
  T.seg_zc = reinterpret_cast<const uint32_t*>(b + L->o_zc);
  L->dsoff[0] = reinterpret_cast<const uint32_t*>(b + L->o_soff[0]);
  L->dsoff[1] = reinterpret_cast<const uint32_t*>(b + L->o_soff[1]);
  T.chunk_sf = reinterpret_cast<const int32_t*>(b + L->o_csf);
  T.chunk_sl = reinterpret_cast<const int32_t*>(b + L->o_csl);
  T.btile = reinterpret_cast<const uint32_t*>(b + L->o_btile);
  T.nbtiles = (int32_t)(L->btile.size() / kBtWords);
  T.d = (int32_t)L->d;
  T.L = L->L;
  T.nchunks = L->nchunks;
  T.nrows = L->nrows;
  T.K = (int32_t)L->K;
  T.nruns = L->nruns;
  T.rk_direct = L->rk_direct ? 1 : 0;
  T.tk_retry = L->tk_retry != 0.0 ? 1 : 0;
  L->bound = true;
  return EF_OK;
}

size_t ef_workspace_bytes(const ef_layout* layout, int op, int32_t W) {
  if (!layout || !layout->valid) return 0;
  switch (op) {
    case EF_OP_TOPK:
    case EF_OP_RANDK: return layout->ws_layout(op).total;
    case EF_OP_RANDBLOCK: return 0;
    case EF_OP_AGG_SPARSE:
      if (W < 1) return 0;
      return align_up((size_t)W * ((size_t)agg_tiles(layout->d) + 1) * 4, kAlign);
    case EF_OP_AGG_BLOCK: return 0;
    case EF_OP_RANDK_PREP:
      // the random-k selection's workspace, then the prepared message's tile table
      return layout->ws_layout(EF_OP_RANDK).total + align_up(((size_t)agg_tiles(layout->d) + 1) * 4, kAlign);
    case EF_OP_AGG_SHARED:
      if (W < 1) return 0;
      // the column sums and one message's tile ranges
      return align_up((size_t)layout->K * 4, kAlign) + align_up(((size_t)agg_tiles(layout->d) + 1) * 4, kAlign);
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
  const dim3 grid((unsigned)((L->d + kRbTile - 1) / kRbTile)), blk(kRbNT);
  if (g_dtype == EF_F32)
    EF_LAUNCH(k_accumulate<0>, grid, blk, 0, S(stream), L->T.d, g, e, acc);
  else
    EF_LAUNCH(k_accumulate<1>, grid, blk, 0, S(stream), L->T.d, g, e, acc);
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

int ef_step_topk_phases(const ef_layout* L, unsigned phases, const void* g, int g_dtype, float* e, uint32_t* idx,
                        float* val, void* ws, size_t ws_bytes, void* stream) {
  EF_TRY(check_bound(L));
  EF_TRY(check_g(g, g_dtype));
  if (!vec_ok(e) || !word_ok(idx) || !word_ok(val) || phases == 0 || (phases & ~EF_PHASE_ALL)) return EF_EINVAL;
  return run_topk(L, g, g_dtype, e, e, idx, val, ws, ws_bytes, stream, phases);
}

// W workers' fused steps in one call (see the header).
int step_batch(int kind, const ef_layout* L, unsigned phases, int32_t W, const void* const* g, int g_dtype,
               float* const* e, const uint64_t* seeds, uint32_t step, uint32_t* idx, float* val, void* ws,
               size_t ws_stride, void* stream) {
  EF_TRY(check_bound(L));
  if (W < 1 || W > 65535) return EF_ERANGE;
  if (phases == 0 || (phases & ~EF_PHASE_ALL)) return EF_EINVAL;
  if (!g || !e || !word_ok(idx) || !word_ok(val)) return EF_EINVAL;
  if (kind == 1 && !seeds) return EF_EINVAL;
  for (int32_t w = 0; w < W; ++w) {
    EF_TRY(check_g(g[w], g_dtype));
    if (!vec_ok(e[w])) return EF_EINVAL;
  }
  if (!ws || !aligned(ws, kAlign) || ws_stride % kAlign) return EF_EINVAL;
  if (ws_stride < ef_workspace_bytes(L, kind == 0 ? EF_OP_TOPK : EF_OP_RANDK, 1)) return EF_EWORKSPACE;
  Steps P;
  P.W = W;
  P.g = g;
  P.g_dtype = g_dtype;
  P.src = const_cast<const float* const*>(e);
  P.e = e;
  P.idx = idx;
  P.val = val;
  P.ws = static_cast<uint8_t*>(ws);
  P.ws_bytes = ws_stride;
  P.ws_stride = ws_stride;
  P.seeds = seeds;
  P.step = step;
  return kind == 0 ? run_select<0>(L, P, phases, stream) : run_select<1>(L, P, phases, stream);
}

int ef_step_topk_batch(const ef_layout* L, unsigned phases, int32_t W, const void* const* g, int g_dtype,
                       float* const* e, uint32_t* idx, float* val, void* ws, size_t ws_stride, void* stream) {
  return step_batch(0, L, phases, W, g, g_dtype, e, nullptr, 0u, idx, val, ws, ws_stride, stream);
}

int ef_step_randk_batch(const ef_layout* L, unsigned phases, int32_t W, const void* const* g, int g_dtype,
                        float* const* e, const uint64_t* seeds, uint32_t step, uint32_t* idx, float* val, void* ws,
                        size_t ws_stride, void* stream) {
  return step_batch(1, L, phases, W, g, g_dtype, e, seeds, step, idx, val, ws, ws_stride, stream);
}

// Random-k prepared ahead: W workers' selections without data (their streaming passes compute
// keys only), the message indices emitted, and each message's tile table after the selection's
// part of its workspace.
static int prepare_randk(const ef_layout* L, int32_t W, const uint64_t* seeds, uint32_t step, uint32_t* idx, void* ws,
                  size_t ws_bytes, size_t ws_stride, void* stream) {
  EF_TRY(check_bound(L));
  if (W < 1 || W > 65535) return EF_ERANGE;
  if (!seeds || !word_ok(idx) || !ws || !aligned(ws, kAlign)) return EF_EINVAL;
  if (ws_bytes < ef_workspace_bytes(L, EF_OP_RANDK_PREP, 1)) return EF_EWORKSPACE;
  std::vector<const float*> none;
  try {
    none.assign((size_t)W, nullptr);
  } catch (const std::bad_alloc&) {
    return EF_ENOMEM;
  }
  Steps P;
  P.W = W;
  P.src = none.data();
  P.idx = idx;
  P.ws = static_cast<uint8_t*>(ws);
  P.ws_bytes = ws_bytes;
  P.ws_stride = ws_stride;
  P.seeds = seeds;
  P.step = step;
  EF_TRY(run_select<1>(L, P, EF_PHASE_ALL, stream));
  const int32_t nt = agg_tiles(L->d);
  const uint32_t blocks = agg_ranges_gx((int32_t)L->K, W);
  uint32_t* ts = reinterpret_cast<uint32_t*>(static_cast<uint8_t*>(ws) + L->ws_layout(EF_OP_RANDK).total);
  if (agg_ranges_big((int32_t)L->K, W))
    EF_LAUNCH(k_agg_ranges<kRangeUBig>, dim3((unsigned)blocks, (unsigned)W), dim3(kNT), 0, S(stream), L->T.d,
              (int32_t)L->K, nt, idx, ts, (uint64_t)(ws_stride / 4), nullptr, 0, nullptr);
  else
    EF_LAUNCH(k_agg_ranges<1>, dim3((unsigned)blocks, (unsigned)W), dim3(kNT), 0, S(stream), L->T.d, (int32_t)L->K,
              nt, idx, ts, (uint64_t)(ws_stride / 4), nullptr, 0, nullptr);
  return launched();
}

static int apply_randk(const ef_layout* L, const void* g, int g_dtype, float* e, const uint32_t* idx, float* val,
                const void* ws, size_t ws_bytes, hipStream_t st) {
  EF_TRY(check_g(g, g_dtype));
  if (!vec_ok(e) || !word_ok(idx) || !word_ok(val) || !ws || !aligned(ws, kAlign)) return EF_EINVAL;
  if (ws_bytes < ef_workspace_bytes(L, EF_OP_RANDK_PREP, 1)) return EF_EWORKSPACE;
  const uint32_t* ts =
      reinterpret_cast<const uint32_t*>(static_cast<const uint8_t*>(ws) + L->ws_layout(EF_OP_RANDK).total);
  const dim3 grid((unsigned)agg_tiles(L->d)), blk(kNT);
  if (g_dtype == EF_F32)
    EF_LAUNCH(k_randk_apply<0>, grid, blk, 0, st, L->T.d, (int32_t)L->K, ts, idx, g, e, val);
  else
    EF_LAUNCH(k_randk_apply<1>, grid, blk, 0, st, L->T.d, (int32_t)L->K, ts, idx, g, e, val);
  return launched();
}

int ef_randk_prepare(const ef_layout* L, uint64_t seed, uint32_t step, uint32_t* idx, void* ws, size_t ws_bytes,
                     void* stream) {
  return prepare_randk(L, 1, &seed, step, idx, ws, ws_bytes, 0, stream);
}

int ef_randk_prepare_batch(const ef_layout* L, int32_t W, const uint64_t* seeds, uint32_t step, uint32_t* idx,
                           void* ws, size_t ws_stride, void* stream) {
  if (ws_stride % kAlign) return EF_EINVAL;
  return prepare_randk(L, W, seeds, step, idx, ws, ws_stride, ws_stride, stream);
}

int ef_step_randk_prepared(const ef_layout* L, const void* g, int g_dtype, float* e, const uint32_t* idx,
                           float* val, const void* ws, size_t ws_bytes, void* stream) {
  EF_TRY(check_bound(L));
  return apply_randk(L, g, g_dtype, e, idx, val, ws, ws_bytes, S(stream));
}

int ef_step_randk_prepared_batch(const ef_layout* L, int32_t W, const void* const* g, int g_dtype, float* const* e,
                                 const uint32_t* idx, float* val, const void* ws, size_t ws_stride, void* stream) {
  EF_TRY(check_bound(L));
  if (W < 1 || W > 65535) return EF_ERANGE;
  if (!g || !e || !word_ok(idx) || !word_ok(val) || ws_stride % kAlign) return EF_EINVAL;
  for (int32_t w = 0; w < W; ++w) {  // every argument before the first launch
    EF_TRY(check_g(g[w], g_dtype));
    if (!vec_ok(e[w])) return EF_EINVAL;
  }
  const uint64_t K = (uint64_t)L->K;
  for (int32_t w = 0; w < W; ++w)
    EF_TRY(apply_randk(L, g[w], g_dtype, e[w], idx + (uint64_t)w * K, val + (uint64_t)w * K,
                       static_cast<const uint8_t*>(ws) + (uint64_t)w * ws_stride, ws_stride, S(stream)));
  return EF_OK;
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

int ef_step_randk_phases(const ef_layout* L, unsigned phases, const void* g, int g_dtype, float* e, uint64_t seed,
                         uint32_t step, uint32_t* idx, float* val, void* ws, size_t ws_bytes, void* stream) {
  EF_TRY(check_bound(L));
  EF_TRY(check_g(g, g_dtype));
  if (!vec_ok(e) || !word_ok(idx) || !word_ok(val) || phases == 0 || (phases & ~EF_PHASE_ALL)) return EF_EINVAL;
  return run_randk(L, g, g_dtype, e, e, seed, step, idx, val, ws, ws_bytes, stream, phases);
}

int compress_randblock(const ef_layout* L, const float* acc, uint64_t seed, uint32_t step, uint32_t* start,
                       float* val, void* stream) {
  EF_TRY(check_bound(L));
  if (!vec_ok(acc) || !word_ok(start) || !word_ok(val)) return EF_EINVAL;
  const unsigned blocks = (unsigned)((L->K + kNT - 1) / kNT);
  EF_LAUNCH(k_randblock_gather, dim3(blocks), dim3(kNT), 0, S(stream), L->T, (int32_t)L->K, acc,
                     (uint32_t)seed, (uint32_t)(seed >> 32), step, start, val);
  return launched();
}

int ef_step_randblock(const ef_layout* L, const void* g, int g_dtype, float* e, uint64_t seed, uint32_t step,
                      uint32_t* start, float* val, void* stream) {
  EF_TRY(check_bound(L));
  EF_TRY(check_g(g, g_dtype));
  if (!vec_ok(e) || !word_ok(start) || !word_ok(val)) return EF_EINVAL;
  const dim3 blk(kRbNT);
  const uint32_t s0 = (uint32_t)seed, s1 = (uint32_t)(seed >> 32);
  if (g_dtype == EF_F32)
    EF_LAUNCH(k_randblock_step<0>, dim3((unsigned)((L->d + rb_tile<0>() - 1) / rb_tile<0>())), blk, 0, S(stream),
              L->T, g, e, s0, s1, step, start, val);
  else
    EF_LAUNCH(k_randblock_step<1>, dim3((unsigned)((L->d + rb_tile<1>() - 1) / rb_tile<1>())), blk, 0, S(stream),
              L->T, g, e, s0, s1, step, start, val);
  return launched();
}

int ef_update(const ef_layout* L, const float* acc, int msg_kind, const uint32_t* m, float* e, void* stream) {
  EF_TRY(check_bound(L));
  if (!vec_ok(acc) || !vec_ok(e) || !word_ok(m)) return EF_EINVAL;
  hipStream_t st = S(stream);
  const unsigned kblocks = (unsigned)((L->K + kNT - 1) / kNT);
  if (msg_kind == EF_MSG_SPARSE) {
    if (e != acc) {
      EF_LAUNCH(k_copy, dim3((unsigned)((L->d + kRbTile - 1) / kRbTile)), dim3(kRbNT), 0, st, L->T.d, acc, e);
      EF_TRY(launched());
    }
    EF_LAUNCH(k_sparse_zero, dim3(kblocks), dim3(kNT), 0, st, L->T.d, (int32_t)L->K, m, e);
    return launched();
  }
  if (msg_kind == EF_MSG_BLOCK) {
    if (e == acc)
      EF_LAUNCH(k_block_zero, dim3(kblocks), dim3(kNT), 0, st, L->T, (int32_t)L->K, m, e);
    else
      EF_LAUNCH(k_block_update, dim3((unsigned)((L->d + kRbTile - 1) / kRbTile)), dim3(kRbNT), 0, st, L->T, acc, m,
                e);
    return launched();
  }
  return EF_EINVAL;
}

}  // extern "C"

namespace {

// The aggregate of W messages through the output stage O (see AggOut).  With `sums` (shared
// coordinates: W = 1 and val holds vW workers' rows), the ranges pass first writes the rows'
// column sums there and the aggregate reads those.
int run_aggregate(const ef_layout* L, int msg_kind, int32_t W, const uint32_t* m, const float* val, const AggOut& O,
                  void* ws, size_t ws_bytes, hipStream_t st, int32_t vW = 0, float* sums = nullptr) {
  const dim3 blk(kNT);
  if (msg_kind == EF_MSG_SPARSE) {
    const size_t need = ef_workspace_bytes(L, EF_OP_AGG_SPARSE, W);
    if (!ws || !aligned(ws, kAlign)) return EF_EINVAL;
    if (ws_bytes < need) return EF_EWORKSPACE;
    const uint32_t blocks = agg_ranges_gx((int32_t)L->K, W);
    uint32_t* ts = reinterpret_cast<uint32_t*>(ws);
    const int32_t nt = agg_tiles(L->d);
    if (agg_ranges_big((int32_t)L->K, W))
      EF_LAUNCH(k_agg_ranges<kRangeUBig>, dim3((unsigned)blocks, (unsigned)W), blk, 0, st, L->T.d, (int32_t)L->K, nt,
                m, ts, (uint64_t)(nt + 1), val, vW, sums);
    else
      EF_LAUNCH(k_agg_ranges<1>, dim3((unsigned)blocks, (unsigned)W), blk, 0, st, L->T.d, (int32_t)L->K, nt, m, ts,
                (uint64_t)(nt + 1), val, vW, sums);
    EF_TRY(launched());
    EF_LAUNCH(k_agg_sparse, dim3((unsigned)nt), dim3(64), 0, st, L->T.d, W, (int32_t)L->K, nt, m,
              sums ? sums : val, ts, O);
    return launched();
  }
  if (msg_kind == EF_MSG_BLOCK) {
    if (L->L == 1) {
      constexpr uint32_t kT1 = 4u * kNT;  // one float4 group per thread
      EF_LAUNCH(k_agg_block1<1>, dim3((unsigned)((L->d + kT1 - 1) / kT1)), blk, 0, st, L->T.d, W, (int32_t)L->K,
                m, val, O);
      return launched();
    }
    EF_LAUNCH(k_agg_block, dim3((unsigned)L->T.nbtiles), blk, 0, st, L->T, W, (int32_t)L->K, m, val, O);
    return launched();
  }
  return EF_EINVAL;
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The address of `scratch` on device dev, resolved once per device with that device current.
int scratch_on(int dev, void** out) {
  if (dev < 0 || dev >= kMaxDevices) return EF_ERANGE;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    int cur = -1;
    EF_TRY(hip_status(hipGetDevice(&cur)));
    if (cur != dev) EF_TRY(hip_status(hipSetDevice(dev)));
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (cur != dev) (void)hipSetDevice(cur);
    EF_TRY(hip_status(e));
    if (!p) return EF_EHIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return EF_OK;
}

}  // namespace

extern "C" {

size_t ef_noalloc_scratch_bytes(void) { return kNoAllocScratch; }

int decompress_aggregate_noalloc(const ef_layout* L, int msg_kind, int32_t W, const uint32_t* m, const float* val,
                                 int average, float* out, void* stream) {
  EF_TRY(check_bound(L));
  if (W < 1 || W > 65535) return EF_ERANGE;
  if (!word_ok(m) || !word_ok(val) || !vec_ok(out)) return EF_EINVAL;
  if (msg_kind != EF_MSG_SPARSE && msg_kind != EF_MSG_BLOCK) return EF_EINVAL;
  if (ef_workspace_bytes(L, msg_kind == EF_MSG_SPARSE ? EF_OP_AGG_SPARSE : EF_OP_AGG_BLOCK, W) > kNoAllocScratch)
    return EF_EWORKSPACE;
  hipStream_t st = S(stream);
  int dev = 0;
  if (st) EF_TRY(hip_status(hipStreamGetDevice(st, &dev)));
  else EF_TRY(hip_status(hipGetDevice(&dev)));
  void* ws = nullptr;
  EF_TRY(scratch_on(dev, &ws));
  const AggOut O{out, nullptr, nullptr, 0.0f, 0.0f, W, average ? 1 : 0};
  return run_aggregate(L, msg_kind, W, m, val, O, ws, kNoAllocScratch, st);
}

int decompress_aggregate(const ef_layout* L, int msg_kind, int32_t W, const uint32_t* m, const float* val,
                         int average, float* out, void* ws, size_t ws_bytes, void* stream) {
  EF_TRY(check_bound(L));
  if (W < 1 || W > 65535) return EF_ERANGE;
  if (!word_ok(m) || !word_ok(val) || !vec_ok(out)) return EF_EINVAL;
  const AggOut O{out, nullptr, nullptr, 0.0f, 0.0f, W, average ? 1 : 0};
  return run_aggregate(L, msg_kind, W, m, val, O, ws, ws_bytes, S(stream));
}

int decompress_aggregate_apply(const ef_layout* L, int msg_kind, int32_t W, const uint32_t* m, const float* val,
                               int average, float* x, float* mom, float beta, float wd, float* out, void* ws,
                               size_t ws_bytes, void* stream) {
  EF_TRY(check_bound(L));
  if (W < 1 || W > 65535) return EF_ERANGE;
  if (!word_ok(m) || !word_ok(val) || !vec_ok(x) || (mom && !vec_ok(mom)) || (out && !vec_ok(out)))
    return EF_EINVAL;
  if (!std::isfinite(beta) || !std::isfinite(wd)) return EF_EINVAL;
  if (mom == x || (out && (out == x || out == mom))) return EF_EINVAL;
  const AggOut O{out, x, mom, beta, wd, W, average ? 1 : 0};
  return run_aggregate(L, msg_kind, W, m, val, O, ws, ws_bytes, S(stream));
}

int decompress_aggregate_shared(const ef_layout* L, int msg_kind, int32_t W, const uint32_t* m, const float* val,
                                int average, float* out, void* ws, size_t ws_bytes, void* stream) {
  EF_TRY(check_bound(L));
  if (W < 1 || W > 65535) return EF_ERANGE;
  if (!word_ok(m) || !word_ok(val) || !vec_ok(out)) return EF_EINVAL;
  if (msg_kind != EF_MSG_SPARSE && msg_kind != EF_MSG_BLOCK) return EF_EINVAL;
  if (!ws || !aligned(ws, kAlign)) return EF_EINVAL;
  if (ws_bytes < ef_workspace_bytes(L, EF_OP_AGG_SHARED, W)) return EF_EWORKSPACE;
  // one message (the shared coordinates) whose values are the column sums of the W workers'
  // values in worker order, divided by W
  hipStream_t st = S(stream);
  float* sum = reinterpret_cast<float*>(ws);
  void* ws1 = reinterpret_cast<uint8_t*>(ws) + align_up((size_t)L->K * 4, kAlign);
  const size_t ws1_bytes = ws_bytes - align_up((size_t)L->K * 4, kAlign);
  const AggOut O{out, nullptr, nullptr, 0.0f, 0.0f, W, average ? 1 : 0};
  if (msg_kind == EF_MSG_SPARSE) return run_aggregate(L, msg_kind, 1, m, val, O, ws1, ws1_bytes, st, W, sum);
  EF_LAUNCH(k_shared_sum, dim3((unsigned)(((size_t)L->K + kNT - 1) / kNT)), dim3(kNT), 0, st, W, (int32_t)L->K, val,
            sum);
  EF_TRY(launched());
  return run_aggregate(L, msg_kind, 1, m, sum, O, ws1, ws1_bytes, st);
}

int ef_dense_average(const ef_layout* L, int32_t W, const float* g, int average, float* out, void* stream) {
  EF_TRY(check_bound(L));
  if (W < 1 || W > 65535) return EF_ERANGE;
  if (!vec_ok(g) || !vec_ok(out)) return EF_EINVAL;
  const size_t groups = ((size_t)L->d + 3) / 4;
  EF_LAUNCH(k_dense_average, dim3((unsigned)(((groups + 1) / 2 + kNT - 1) / kNT)), dim3(kNT), 0, S(stream), L->T.d, W, g,
            average ? 1 : 0, out);
  return launched();
}

}  // extern "C"
