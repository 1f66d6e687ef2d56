// Seeded synthetic graph generator shared by the tests, the benchmark and the
// oracle's callers.  It builds the CSR of A + I (adjacency plus one self-loop
// per node) for an undirected power-law graph drawn from the R-MAT model
// (Chakrabarti, Zhan, Faloutsos, SDM 2004).  It contains no part of the
// binarized-GCN arithmetic: no normalisation, no signs, no scales.
//
// Determinism: every random number is a pure function of (seed, counter)
// through the SplitMix64 finaliser (Steele, Lea, Flood, OOPSLA 2014), so the
// graph is identical for any thread count and any candidate batch size.
//
// Recipe (one call):
//   1. Candidate edge e (e = 0, 1, 2, ...) picks, at each of S = ceil(log2 n)
//      levels, one quadrant with probabilities (a, b, c, 1-a-b-c); the levels
//      give the bits of (u, v).  Candidates with u >= n, v >= n or u == v are
//      rejected.
//   2. Undirected canonical key (min, max); the first T distinct keys in
//      candidate order are kept, so the edge count is exact.
//   3. A seeded random relabelling of the node ids (so R-MAT's id locality
//      does not flatter caches), both directions of every edge, one
//      self-loop per node, CSR with column indices sorted inside each row.

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <memory>
#include <numeric>
#include <vector>
#include <omp.h>

namespace {

inline uint64_t mix64(uint64_t z) {
  z += 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Stream base: one finaliser pass over (seed, stream); draws then cost one
// more pass each.
inline uint64_t stream_base(uint64_t seed, uint64_t stream) {
  return mix64(seed ^ (stream * 0xD1B54A32D192ED03ull));
}

inline uint64_t draw(uint64_t base, uint64_t ctr) { return mix64(base + ctr); }

struct Rmat {
  int64_t n;
  int scale;
  uint32_t ta, tb, tc;  // cumulative thresholds on a 16-bit draw
  uint64_t base;  // stream_base(seed, 1)

  // Returns false for a rejected candidate.
  bool edge(uint64_t e, int64_t* lo, int64_t* hi) const {
    uint64_t u = 0, v = 0;
    uint64_t bits = 0;
    for (int l = 0; l < scale; ++l) {
      if ((l & 3) == 0) bits = draw(base, e * 8 + (uint64_t)(l >> 2));
      uint32_t r = (uint32_t)(bits & 0xFFFF);
      bits >>= 16;
      uint64_t ub = r >= tb;                       // quadrants c, d
      uint64_t vb = (r >= ta && r < tb) || r >= tc;  // quadrants b, d
      u |= ub << l;
      v |= vb << l;
    }
    if ((int64_t)u >= n || (int64_t)v >= n || u == v) return false;
    *lo = (int64_t)std::min(u, v);
    *hi = (int64_t)std::max(u, v);
    return true;
  }
};

}  // namespace

extern "C" {

// Number of directed entries of A + I for T undirected edges.
int64_t wl_nnz(int64_t n, int64_t n_undirected) { return 2 * n_undirected + n; }

// Builds CSR(A + I).  rowptr has n + 1 entries, colidx has 2T + n entries.
// Returns 0 on success, -1 on bad arguments, -2 if the candidate budget
// (64 x T + 2^20) ran out before T distinct edges were found.
int wl_rmat_csr(int64_t n, int64_t n_undirected, uint64_t seed, double a,
                double b, double c, int64_t* rowptr, int32_t* colidx) {
  if (n <= 1 || n_undirected < 0 || n > (int64_t(1) << 31) - 1) return -1;
  if (n_undirected > n * (n - 1) / 2) return -1;
  Rmat g;
  g.n = n;
  g.scale = 0;
  while ((int64_t(1) << g.scale) < n) ++g.scale;
  g.ta = (uint32_t)std::lround(a * 65536.0);
  g.tb = (uint32_t)std::lround((a + b) * 65536.0);
  g.tc = (uint32_t)std::lround((a + b + c) * 65536.0);
  g.base = stream_base(seed, 1);
  const int64_t T = n_undirected;

  // 1-2: first T distinct canonical edges in candidate order.
  std::vector<uint64_t> keep_keys;  // the T kept keys, candidate order
  if (T > 0) {
    uint64_t ncand = (uint64_t)T * 3 + 4096;
    const uint64_t budget = (uint64_t)T * 64 + (1u << 20);
    const int nt = omp_get_max_threads();
    for (;;) {
      const int64_t nc = (int64_t)ncand;
      // Arrays are first touched inside the parallel loops (no serial
      // zero-fill); a rejected candidate has key ~0.
      std::unique_ptr<uint64_t[]> key(new uint64_t[nc]);
      std::unique_ptr<uint8_t[]> first(new uint8_t[nc]);
#pragma omp parallel for schedule(static)
      for (int64_t e = 0; e < nc; ++e) {
        int64_t lo, hi;
        key[e] = g.edge((uint64_t)e, &lo, &hi)
                     ? (uint64_t)lo * (uint64_t)n + (uint64_t)hi
                     : ~0ull;
        first[e] = 0;
      }
      // Group equal keys: bucket candidates by a hash of the key (parallel
      // counting sort; R-MAT keys are far too skewed to bucket by their high
      // bits), then sort each bucket by (key, index).  The kept set does not
      // depend on the thread count.
      const int nb_log = 10;
      const int nb = 1 << nb_log;
      const int shift = 64 - nb_log;
      std::vector<int64_t> tc((size_t)nt * nb, 0);
#pragma omp parallel num_threads(nt)
      {
        const int t = omp_get_thread_num();
        const int64_t lo = nc * t / nt, hi = nc * (t + 1) / nt;
        int64_t* c = &tc[(size_t)t * nb];
        for (int64_t e = lo; e < hi; ++e)
          if (key[e] != ~0ull) c[mix64(key[e]) >> shift]++;
      }
      std::vector<int64_t> cnt(nb + 1, 0);
      {
        int64_t run = 0;
        for (int bkt = 0; bkt < nb; ++bkt) {
          cnt[bkt] = run;
          for (int t = 0; t < nt; ++t) {
            int64_t v = tc[(size_t)t * nb + bkt];
            tc[(size_t)t * nb + bkt] = run;
            run += v;
          }
        }
        cnt[nb] = run;
      }
      const int64_t nok = cnt[nb];
      std::unique_ptr<std::pair<uint64_t, uint64_t>[]> kv(
          new std::pair<uint64_t, uint64_t>[nok]);
#pragma omp parallel num_threads(nt)
      {
        const int t = omp_get_thread_num();
        const int64_t lo = nc * t / nt, hi = nc * (t + 1) / nt;
        int64_t* c = &tc[(size_t)t * nb];
        for (int64_t e = lo; e < hi; ++e)
          if (key[e] != ~0ull) kv[c[mix64(key[e]) >> shift]++] = {key[e], (uint64_t)e};
      }
#pragma omp parallel for schedule(dynamic, 1)
      for (int bkt = 0; bkt < nb; ++bkt) {
        auto* b0 = kv.get() + cnt[bkt];
        auto* b1 = kv.get() + cnt[bkt + 1];
        std::sort(b0, b1);
        for (auto* p = b0; p < b1; ++p)
          if (p == b0 || p->first != (p - 1)->first) first[p->second] = 1;
      }
      kv.reset();
      // Per-thread counts of first occurrences, then the first T in order.
      std::vector<int64_t> fc(nt + 1, 0);
#pragma omp parallel num_threads(nt)
      {
        const int t = omp_get_thread_num();
        const int64_t lo = nc * t / nt, hi = nc * (t + 1) / nt;
        int64_t h = 0;
        for (int64_t e = lo; e < hi; ++e) h += first[e];
        fc[t + 1] = h;
      }
      for (int t = 0; t < nt; ++t) fc[t + 1] += fc[t];
      if (fc[nt] >= T) {
        keep_keys.resize(T);
#pragma omp parallel num_threads(nt)
        {
          const int t = omp_get_thread_num();
          const int64_t lo = nc * t / nt, hi = nc * (t + 1) / nt;
          int64_t o = fc[t];
          for (int64_t e = lo; e < hi && o < T; ++e)
            if (first[e]) keep_keys[o++] = key[e];
        }
        break;
      }
      if (ncand >= budget) return -2;
      ncand = std::min(budget, ncand * 2);
    }
  }

  // 3a: seeded relabelling pi (argsort of per-node random keys).
  std::vector<int64_t> pi(n);
  {
    const uint64_t perm_base = stream_base(seed, 2);
    std::vector<std::pair<uint64_t, int64_t>> r(n);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; ++i) r[i] = {draw(perm_base, (uint64_t)i), i};
    std::sort(r.begin(), r.end());
    for (int64_t i = 0; i < n; ++i) pi[r[i].second] = i;
  }

  // 3b: degrees of A + I, row pointers.
  std::vector<std::atomic<int64_t>> deg(n);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) deg[i].store(1, std::memory_order_relaxed);
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < T; ++t) {
    int64_t lo = (int64_t)(keep_keys[t] / (uint64_t)n);
    int64_t hi = (int64_t)(keep_keys[t] % (uint64_t)n);
    deg[pi[lo]].fetch_add(1, std::memory_order_relaxed);
    deg[pi[hi]].fetch_add(1, std::memory_order_relaxed);
  }
  rowptr[0] = 0;
  for (int64_t i = 0; i < n; ++i) rowptr[i + 1] = rowptr[i] + deg[i].load();

  // 3c: fill (self-loop first), then sort each row.
  std::vector<std::atomic<int64_t>> fill(n);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    colidx[rowptr[i]] = (int32_t)i;
    fill[i].store(rowptr[i] + 1, std::memory_order_relaxed);
  }
#pragma omp parallel for schedule(static)
  for (int64_t t = 0; t < T; ++t) {
    int64_t a0 = pi[(int64_t)(keep_keys[t] / (uint64_t)n)];
    int64_t b0 = pi[(int64_t)(keep_keys[t] % (uint64_t)n)];
    colidx[fill[a0].fetch_add(1, std::memory_order_relaxed)] = (int32_t)b0;
    colidx[fill[b0].fetch_add(1, std::memory_order_relaxed)] = (int32_t)a0;
  }
#pragma omp parallel for schedule(dynamic, 256)
  for (int64_t i = 0; i < n; ++i)
    std::sort(colidx + rowptr[i], colidx + rowptr[i + 1]);
  return 0;
}

}  // extern "C"
