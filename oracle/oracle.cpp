// PinSage CPU oracle — TEST INFRASTRUCTURE ONLY.
//
// A plain, slow, obviously-correct CPU statement of what the PinSage hot path
// computes (Ying et al., "Graph Convolutional Neural Networks for Web-Scale
// Recommender Systems", KDD 2018). Only the test-suite, the smoke check and the
// benchmark's CPU-baseline leg may load this library; the product path never
// does. It shares no code, header or constant table with the GPU library.
//
// Every function below follows one passage of the paper, cited in its comment:
//   * Philox4x32-10 .......... Salmon et al., SC'11 ("Parallel random numbers:
//                              as easy as 1, 2, 3"), Sec. 3.2 + Table 2.
//   * random walks / counts .. Sec. 3.2, "Importance-based neighborhoods".
//   * top-T + L1 weights ..... Sec. 3.2, same paragraph and "importance pooling".
//   * CONVOLVE ............... Sec. 3.2, Algorithm 1 (lines 1-3).
//   * stacked layers ......... Sec. 3.2, "Stacking convolutions".
//   * layer-wise inference ... Sec. 3.4 (project every pin once, then pool).
//   * MINIBATCH sets + loop .. Sec. 3.2, Algorithm 2 (sampling and embedding).
//   * max-margin loss ........ Sec. 3.3, Eq. (1).
//   * aggregators gamma ...... importance pooling (Sec. 3.2), and the element-wise
//                              mean and max of the compared variants (Sec. 4).
//   * output dense layers .... Algorithm 2, final loop: z = G2 ReLU(G1 h + g).
//   * hard negative items .... Sec. 3.3 (PPR rank window, sampled).
//   * graph neighbourhoods ... Sec. 3.4 (MapReduce: boards pool their pins,
//                              pins their boards; long rows sampled).
//
// Readings of points the paper leaves open are listed in the repository's
// design notes; the ones that change arithmetic are restated at each function.
// All floating point is fp64 except the importance weights, which the method
// stores as fp32 (one fp32 division c/S per weight).
//
// Parity pins: every exported function is pinned by a CPU test against an
// independent statement (published known-answer vectors, a library routine,
// closed-form expectations, brute force or a special case); see tests/.

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <map>
#include <set>
#include <thread>
#include <utility>
#include <vector>

namespace {

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon et al., SC'11). One round maps the 128-bit counter
// (c0,c1,c2,c3) with 64-bit key (k0,k1) to
//   (hi(M1*c2) ^ c1 ^ k0,  lo(M1*c2),  hi(M0*c0) ^ c3 ^ k1,  lo(M0*c0))
// and the key is bumped by the Weyl constants between rounds.
// ---------------------------------------------------------------------------
const uint32_t kPhiloxM0 = 0xD2511F53u;
const uint32_t kPhiloxM1 = 0xCD9E8D57u;
const uint32_t kWeyl0 = 0x9E3779B9u;  // golden ratio
const uint32_t kWeyl1 = 0xBB67AE85u;  // sqrt(3) - 1

void philox4x32_10(const uint32_t in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c[4] = {in[0], in[1], in[2], in[3]};
  uint32_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; ++round) {
    uint64_t p0 = (uint64_t)kPhiloxM0 * (uint64_t)c[0];
    uint64_t p1 = (uint64_t)kPhiloxM1 * (uint64_t)c[2];
    uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    uint32_t n0 = hi1 ^ c[1] ^ k0;
    uint32_t n1 = lo1;
    uint32_t n2 = hi0 ^ c[3] ^ k1;
    uint32_t n3 = lo0;
    c[0] = n0; c[1] = n1; c[2] = n2; c[3] = n3;
    k0 += kWeyl0;
    k1 += kWeyl1;
  }
  out[0] = c[0]; out[1] = c[1]; out[2] = c[2]; out[3] = c[3];
}

// The random word used at edge step s of walk w from source u.
// Stream layout (a reading; the paper does not fix one): counter
// (u, w, s/4, 0), key (lo32(seed), hi32(seed)); step s uses output word s%4.
uint32_t walk_word(uint64_t seed, uint32_t u, uint32_t w, uint32_t s) {
  uint32_t ctr[4] = {u, w, s / 4u, 0u};
  uint32_t key[2] = {(uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32)};
  uint32_t out[4];
  philox4x32_10(ctr, key, out);
  return out[s % 4u];
}

struct Graph {
  const int64_t* off;   // [num_nodes + 1]
  const int32_t* col;   // [off[num_nodes]]
  int64_t num_pins;     // pins are ids [0, num_pins)
  int64_t num_nodes;    // boards are ids [num_pins, num_nodes)
};

// Sec. 3.2, importance-based neighbourhoods: simulate random walks from u and
// record every pin the walk lands on. Readings: each walk is unbiased (the next
// node is a uniformly chosen CSR neighbour; the draw maps the 32-bit word r to
// index floor(r*deg / 2^32)), a walk ends after `hops` landings on a pin, after
// 2*hops edge steps, or at a node with no edges; the source itself is not
// recorded. Appends visited pin ids to `visits`; returns edge steps taken.
int64_t walk_from(const Graph& g, uint64_t seed, int64_t u, int walks, int hops,
                  std::vector<int32_t>& visits) {
  int64_t steps = 0;
  for (int w = 0; w < walks; ++w) {
    int64_t cur = u;
    int landed = 0;
    int s = 0;
    while (landed < hops && s < 2 * hops) {
      int64_t deg = g.off[cur + 1] - g.off[cur];
      if (deg <= 0) break;
      uint32_t r = walk_word(seed, (uint32_t)u, (uint32_t)w, (uint32_t)s);
      int64_t j = (int64_t)(((uint64_t)r * (uint64_t)deg) >> 32);
      cur = g.col[g.off[cur] + j];
      ++s;
      if (cur < g.num_pins) {
        ++landed;
        if (cur != u) visits.push_back((int32_t)cur);
      }
    }
    steps += s;
  }
  return steps;
}

// Sec. 3.2: the neighbourhood is the T pins with the highest visit counts;
// importance pooling weights them by their L1-normalised counts. Readings:
// ties are broken by the lower node id, and the L1 normalisation runs over the
// kept T counts, so the weights of a row sum to one (the weighted mean is the
// same under either normalisation). Rows with fewer than T distinct pins are
// padded with (-1, 0, 0.0f).
// The distinct visited pins as (count, id), in rank order: more visits
// first, ties to the lower id.
std::vector<std::pair<int64_t, int32_t>> ranked_pins(const std::vector<int32_t>& visits) {
  std::map<int32_t, int64_t> counts;
  for (int32_t v : visits) counts[v] += 1;
  std::vector<std::pair<int64_t, int32_t>> order;  // (count, id)
  for (const auto& kv : counts) order.push_back({kv.second, kv.first});
  std::sort(order.begin(), order.end(),
            [](const std::pair<int64_t, int32_t>& a, const std::pair<int64_t, int32_t>& b) {
              if (a.first != b.first) return a.first > b.first;  // more visits first
              return a.second < b.second;                        // then lower id
            });
  return order;
}

void select_top_t(const std::vector<int32_t>& visits, int T, int32_t* idx, uint16_t* cnt,
                  float* wts) {
  const std::vector<std::pair<int64_t, int32_t>> order = ranked_pins(visits);
  int keep = (int)std::min<size_t>((size_t)T, order.size());
  int64_t total = 0;
  for (int t = 0; t < keep; ++t) total += order[t].first;
  for (int t = 0; t < T; ++t) {
    if (t < keep) {
      idx[t] = order[t].second;
      cnt[t] = (uint16_t)order[t].first;
      float c = (float)order[t].first;
      float s = (float)total;
      wts[t] = c / s;  // one IEEE fp32 division, round-to-nearest-even
    } else {
      idx[t] = -1;
      cnt[t] = 0;
      wts[t] = 0.0f;
    }
  }
}

template <typename F>
void parallel_rows(int64_t n, int nthreads, F fn) {
  if (nthreads <= 1 || n < 2) {
    fn((int64_t)0, n);
    return;
  }
  std::vector<std::thread> pool;
  int64_t per = (n + nthreads - 1) / nthreads;
  for (int t = 0; t < nthreads; ++t) {
    int64_t lo = t * per, hi = std::min(n, lo + per);
    if (lo >= hi) break;
    pool.emplace_back([=]() { fn(lo, hi); });
  }
  for (auto& th : pool) th.join();
}

// Algorithm 1, line 1 for one neighbour: ReLU(Q h_v + q), Q is [m x d_in].
void transform_row(const double* h, int d_in, const double* Q, const double* q, int m,
                   double* out) {
  for (int i = 0; i < m; ++i) {
    double acc = 0.0;
    for (int j = 0; j < d_in; ++j) acc += Q[(int64_t)i * d_in + j] * h[j];
    acc += q[i];
    out[i] = acc > 0.0 ? acc : 0.0;
  }
}

// Algorithm 1, lines 2-3: z = ReLU(W concat(h_u, n_u) + w); z / ||z||_2.
// W is [d_out x (d_in + m)]: the first d_in columns multiply the node's own
// vector, the remaining m columns multiply the pooled neighbourhood vector.
// A zero z (all pre-activations <= 0) stays zero (the paper divides without a
// guard; this case does not arise with the workloads here).
void combine_row(const double* h_self, int d_in, const double* n_u, int m, const double* W,
                 const double* w, int d_out, double* out) {
  const int K = d_in + m;
  double sq = 0.0;
  for (int o = 0; o < d_out; ++o) {
    double acc = 0.0;
    for (int j = 0; j < d_in; ++j) acc += W[(int64_t)o * K + j] * h_self[j];
    for (int j = 0; j < m; ++j) acc += W[(int64_t)o * K + d_in + j] * n_u[j];
    acc += w[o];
    double z = acc > 0.0 ? acc : 0.0;
    out[o] = z;
    sq += z * z;
  }
  double norm = std::sqrt(sq);
  for (int o = 0; o < d_out; ++o) out[o] = norm > 0.0 ? out[o] / norm : 0.0;
}

// The aggregator gamma of Algorithm 1, line 1, over the transformed
// neighbours of one node, taken in rank order t = 0, 1, ... (ids < 0 are
// padding and are skipped):
//   mode 0, importance pooling (Sec. 3.2): sum_t alpha_t * P_t, alpha the
//           node's normalised visit counts;
//   mode 1, mean (Sec. 4, gamma = mean): (1 / #neighbours) * sum_t P_t;
//   mode 2, max (Sec. 4, gamma = max): element-wise max over the P_t.
// An empty neighbourhood gives the zero vector in every mode.
template <typename RowOf>
void pool_row(int mode, const int32_t* ids, const float* alpha, int T, RowOf row_of, int m,
              double* n_u) {
  int count = 0;
  for (int t = 0; t < T; ++t)
    if (ids[t] >= 0) ++count;
  for (int i = 0; i < m; ++i) n_u[i] = 0.0;
  if (count == 0) return;
  if (mode == 2) {
    bool first = true;
    for (int t = 0; t < T; ++t) {
      if (ids[t] < 0) continue;
      const double* pv = row_of(ids[t]);
      for (int i = 0; i < m; ++i) n_u[i] = first ? pv[i] : std::max(n_u[i], pv[i]);
      first = false;
    }
    return;
  }
  for (int t = 0; t < T; ++t) {
    if (ids[t] < 0) continue;
    const double a = mode == 1 ? 1.0 / (double)count : (double)alpha[t];
    const double* pv = row_of(ids[t]);
    for (int i = 0; i < m; ++i) n_u[i] += a * pv[i];
  }
}

}  // namespace

extern "C" {

int orc_version(void) { return 2; }

// Philox4x32-10 block function, exposed for known-answer tests.
void orc_philox4x32_10(const uint32_t* ctr, const uint32_t* key, uint32_t* out) {
  philox4x32_10(ctr, key, out);
}

uint32_t orc_walk_word(uint64_t seed, uint32_t u, uint32_t w, uint32_t s) {
  return walk_word(seed, u, w, s);
}

// Raw visit list of one source (for brute-force checks of the selection step).
// visits_out must hold walks*hops entries; returns the number written, and the
// edge steps taken in *steps.
int64_t orc_walk_visits(const int64_t* off, const int32_t* col, int64_t num_pins,
                        int64_t num_nodes, uint64_t seed, int64_t u, int walks, int hops,
                        int32_t* visits_out, int64_t* steps) {
  Graph g{off, col, num_pins, num_nodes};
  std::vector<int32_t> v;
  int64_t s = walk_from(g, seed, u, walks, hops, v);
  for (size_t i = 0; i < v.size(); ++i) visits_out[i] = v[i];
  if (steps) *steps = s;
  return (int64_t)v.size();
}

// Importance neighbourhoods (Sec. 3.2) for sources[0..num_sources), or for
// every node when sources is NULL. Outputs are [num_sources x T], row r
// belonging to sources[r]. *total_steps receives the edge steps of all walks.
void orc_build_neighborhoods(const int64_t* off, const int32_t* col, int64_t num_pins,
                             int64_t num_nodes, uint64_t seed, int walks, int hops, int T,
                             const int32_t* sources, int64_t num_sources, int32_t* idx,
                             uint16_t* cnt, float* wts, int64_t* total_steps, int nthreads) {
  Graph g{off, col, num_pins, num_nodes};
  std::vector<int64_t> steps_per_thread(std::max(1, nthreads), 0);
  std::vector<int64_t> chunk_steps;
  int nt = std::max(1, nthreads);
  int64_t per = (num_sources + nt - 1) / nt;
  std::vector<std::thread> pool;
  for (int t = 0; t < nt; ++t) {
    int64_t lo = t * per, hi = std::min(num_sources, lo + per);
    if (lo >= hi) break;
    auto body = [&, t, lo, hi]() {
      std::vector<int32_t> visits;
      int64_t acc = 0;
      for (int64_t r = lo; r < hi; ++r) {
        int64_t u = sources ? (int64_t)sources[r] : r;
        visits.clear();
        acc += walk_from(g, seed, u, walks, hops, visits);
        select_top_t(visits, T, idx + r * T, cnt + r * T, wts + r * T);
      }
      steps_per_thread[t] = acc;
    };
    if (nt == 1) body(); else pool.emplace_back(body);
  }
  for (auto& th : pool) th.join();
  int64_t total = 0;
  for (int64_t s : steps_per_thread) total += s;
  if (total_steps) *total_steps = total;
}

// Sec. 3.4, MapReduce inference: a board's embedding pools the pins it holds
// and, one layer up, a pin's pools its boards (the graph's own adjacency, with
// neighbours "sampled"). Readings: node u's neighbourhood is its CSR row when
// the row has at most T entries (each once); a longer row is sampled with T
// independent draws, draw j taking word 0 of Philox4x32-10 at counter
// (u, j, 0, 2) under the key (lo32(seed), hi32(seed)) and picking row position
// floor(r * deg / 2^32). Entries outside [0, num_nodes) are dropped. The table
// row lists the distinct ids ascending with their multiplicities; the weights
// are multiplicity / (entries kept), one fp32 division (the degree-normalised
// mean of the row or of the sample). Padding: -1, 0, 0.
void orc_graph_neighborhoods(const int64_t* off, const int32_t* col, int64_t num_nodes,
                             uint64_t seed, int T, const int32_t* sources, int64_t num_sources,
                             int32_t* idx, uint16_t* cnt, float* wts, int nthreads) {
  const uint32_t key[2] = {(uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32)};
  parallel_rows(num_sources, nthreads, [&](int64_t lo, int64_t hi) {
    std::vector<int32_t> picked;
    for (int64_t r = lo; r < hi; ++r) {
      const int64_t u = sources ? (int64_t)sources[r] : r;
      for (int t = 0; t < T; ++t) {
        idx[r * T + t] = -1;
        cnt[r * T + t] = 0;
        wts[r * T + t] = 0.0f;
      }
      if (u < 0 || u >= num_nodes) continue;
      const int64_t b = off[u], deg = off[u + 1] - off[u];
      picked.clear();
      if (deg <= T) {
        for (int64_t i = 0; i < deg; ++i) picked.push_back(col[b + i]);
      } else {
        for (int j = 0; j < T; ++j) {
          const uint32_t ctr[4] = {(uint32_t)u, (uint32_t)j, 0u, 2u};
          uint32_t rr[4];
          philox4x32_10(ctr, key, rr);
          picked.push_back(col[b + (int64_t)(((uint64_t)rr[0] * (uint64_t)deg) >> 32)]);
        }
      }
      std::map<int32_t, int64_t> mult;
      int64_t kept = 0;
      for (int32_t v : picked)
        if (v >= 0 && (int64_t)v < num_nodes) {
          mult[v] += 1;
          ++kept;
        }
      int t = 0;
      for (const auto& kv : mult) {  // ascending id
        idx[r * T + t] = kv.first;
        cnt[r * T + t] = (uint16_t)kv.second;
        wts[r * T + t] = (float)kv.second / (float)kept;
        ++t;
      }
    }
  });
}

// One CONVOLVE layer over a set of output rows, in the layer-wise dataflow of
// Sec. 3.4: rows [0, n_transform) of h_in are projected once each with
// Algorithm 1 line 1, then every output row pools its neighbours (importance
// pooling: sum_t alpha_t * P[idx_t], Sec. 3.2) and applies lines 2-3.
// h_out row r uses h_in row self_rows[r] (or r when self_rows is NULL).
// Neighbour ids < 0 are padding and are skipped.
void orc_convolve_layer(const double* h_in, int64_t n_in, int d_in, int64_t n_transform,
                        const double* Q, const double* q, int m, const double* W,
                        const double* w, int d_out, const int32_t* idx, const float* wts, int T,
                        const int64_t* self_rows, int64_t n_out, double* h_out, int nthreads,
                        int pool) {
  (void)n_in;
  std::vector<double> P((size_t)n_transform * (size_t)m);
  parallel_rows(n_transform, nthreads, [&](int64_t lo, int64_t hi) {
    for (int64_t v = lo; v < hi; ++v)
      transform_row(h_in + v * d_in, d_in, Q, q, m, P.data() + v * m);
  });
  parallel_rows(n_out, nthreads, [&](int64_t lo, int64_t hi) {
    std::vector<double> n_u((size_t)m);
    for (int64_t r = lo; r < hi; ++r) {
      pool_row(pool, idx + r * T, wts + r * T, T,
               [&](int32_t v) { return P.data() + (int64_t)v * m; }, m, n_u.data());
      int64_t self = self_rows ? self_rows[r] : r;
      combine_row(h_in + self * d_in, d_in, n_u.data(), m, W, w, d_out, h_out + r * d_out);
    }
  });
}

// Sec. 3.3, hard negative items: the pins are ranked by their Personalized
// PageRank score with respect to the query, and items at ranks in a window
// (the paper: 2000-5000) are sampled at random. Readings: the scores are the
// visit counts of the Sec. 3.2 walks from the query (walks, hops and seed of
// their own), ranked like the neighbourhoods (count descending, ties to the
// lower id, the query itself excluded); the window is [rank_lo, rank_hi),
// 0-based, cut at the number of ranked pins n_r; draw j for query q is word 0
// of Philox4x32-10 at counter (q, j, 0, 1) under the walk key, mapped to
// window position floor(r * n / 2^32), n = min(rank_hi, n_r) - rank_lo
// (independent draws, with replacement). Without a window (n <= 0), or for a
// query id outside the graph, the k entries are -1.
void orc_hard_negatives(const int64_t* off, const int32_t* col, int64_t num_pins,
                        int64_t num_nodes, uint64_t seed, int walks, int hops,
                        const int32_t* queries, int64_t num_queries, int rank_lo, int rank_hi,
                        int k, int32_t* out, int nthreads) {
  Graph g{off, col, num_pins, num_nodes};
  const uint32_t key[2] = {(uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32)};
  parallel_rows(num_queries, nthreads, [&](int64_t lo, int64_t hi) {
    std::vector<int32_t> visits;
    for (int64_t i = lo; i < hi; ++i) {
      const int64_t q = queries[i];
      for (int j = 0; j < k; ++j) out[i * k + j] = -1;
      if (q < 0 || q >= num_nodes) continue;
      visits.clear();
      walk_from(g, seed, q, walks, hops, visits);
      const auto order = ranked_pins(visits);
      const int64_t top = std::min<int64_t>(rank_hi, (int64_t)order.size());
      const int64_t n = top - rank_lo;
      if (n <= 0) continue;
      for (int j = 0; j < k; ++j) {
        const uint32_t ctr[4] = {(uint32_t)q, (uint32_t)j, 0u, 1u};
        uint32_t r[4];
        philox4x32_10(ctr, key, r);
        const int64_t pos = (int64_t)(((uint64_t)r[0] * (uint64_t)n) >> 32);
        out[i * k + j] = order[rank_lo + pos].second;
      }
    }
  });
}

// Algorithm 2, sampling part: S^(K) = M; S^(k-1) = S^(k) united with N(u) for
// every u in S^(k). N(u) is read from a neighbourhood table with one row per
// node (nbr_idx[u*T + t], padding < 0). Writes the sorted node ids of S^(k)
// for k = 0..K into `sets` (concatenated, S^(0) first) and their sizes into
// set_sizes[0..K]. Returns the total length, or -(required length) when
// `cap` is too small (nothing written then).
int64_t orc_minibatch_sets(const int32_t* targets, int64_t num_targets, int K,
                           const int32_t* nbr_idx, int T, int64_t* set_sizes, int32_t* sets,
                           int64_t cap) {
  std::vector<std::set<int32_t>> S(K + 1);
  for (int64_t i = 0; i < num_targets; ++i) S[K].insert(targets[i]);
  for (int k = K; k >= 1; --k) {
    S[k - 1] = S[k];
    for (int32_t u : S[k])
      for (int t = 0; t < T; ++t) {
        int32_t v = nbr_idx[(int64_t)u * T + t];
        if (v >= 0) S[k - 1].insert(v);
      }
  }
  int64_t total = 0;
  for (int k = 0; k <= K; ++k) total += (int64_t)S[k].size();
  if (total > cap) return -total;
  int64_t pos = 0;
  for (int k = 0; k <= K; ++k) {
    set_sizes[k] = (int64_t)S[k].size();
    for (int32_t v : S[k]) sets[pos++] = v;
  }
  return total;
}

}  // extern "C"

namespace {

// Algorithm 2, embedding part (lines 7-13), shared by the full-table and the
// sampled variants below. `x_row(v)` gives h^(0)_v = x_v and `nbr_row(u)` the
// (ids, weights) of N(u); S holds the sorted sets S^(0..K). Each neighbour's
// Algorithm-1 line-1 vector depends only on (k, v), so it is evaluated once
// per distinct v within a layer.
template <typename XRow, typename NbrRow>
void minibatch_embed_impl(const int32_t* targets, int64_t num_targets, int K,
                          const std::vector<std::vector<int32_t>>& S, XRow x_row, int d0,
                          NbrRow nbr_row, int T, const double* const* Qs, const double* const* qs,
                          const int* ms, const double* const* Ws, const double* const* ws,
                          const int* d_outs, const int* pools, double* out, int nthreads) {
  std::map<int32_t, int64_t> pos_prev;  // node -> row in h_prev
  std::vector<double> h_prev((size_t)S[0].size() * d0);
  for (size_t i = 0; i < S[0].size(); ++i) {
    pos_prev[S[0][i]] = (int64_t)i;
    std::memcpy(h_prev.data() + i * d0, x_row(S[0][i]), sizeof(double) * d0);
  }
  int d_prev = d0;
  for (int k = 1; k <= K; ++k) {
    const int m = ms[k - 1], d_out = d_outs[k - 1];
    const double* Q = Qs[k - 1];
    const double* q = qs[k - 1];
    const double* W = Ws[k - 1];
    const double* w = ws[k - 1];
    std::vector<int32_t> need;
    {
      std::set<int32_t> ns;
      for (int32_t u : S[k]) {
        const int32_t* ids = nbr_row(u).first;
        for (int t = 0; t < T; ++t)
          if (ids[t] >= 0) ns.insert(ids[t]);
      }
      need.assign(ns.begin(), ns.end());
    }
    std::map<int32_t, int64_t> pos_need;
    for (size_t i = 0; i < need.size(); ++i) pos_need[need[i]] = (int64_t)i;
    std::vector<double> Pn(need.size() * (size_t)m);
    parallel_rows((int64_t)need.size(), nthreads, [&](int64_t lo, int64_t hi) {
      for (int64_t i = lo; i < hi; ++i)
        transform_row(h_prev.data() + pos_prev.at(need[i]) * d_prev, d_prev, Q, q, m,
                      Pn.data() + i * m);
    });
    std::vector<double> h_next(S[k].size() * (size_t)d_out);
    parallel_rows((int64_t)S[k].size(), nthreads, [&](int64_t lo, int64_t hi) {
      std::vector<double> n_u((size_t)m);
      for (int64_t i = lo; i < hi; ++i) {
        int32_t u = S[k][i];
        const auto row = nbr_row(u);
        pool_row(pools ? pools[k - 1] : 0, row.first, row.second, T,
                 [&](int32_t v) { return Pn.data() + pos_need.at(v) * m; }, m, n_u.data());
        combine_row(h_prev.data() + pos_prev.at(u) * d_prev, d_prev, n_u.data(), m, W, w,
                    d_out, h_next.data() + i * d_out);
      }
    });
    std::map<int32_t, int64_t> pos_next;
    for (size_t i = 0; i < S[k].size(); ++i) pos_next[S[k][i]] = (int64_t)i;
    h_prev.swap(h_next);
    pos_prev.swap(pos_next);
    d_prev = d_out;
  }
  for (int64_t i = 0; i < num_targets; ++i)
    std::memcpy(out + i * d_prev, h_prev.data() + pos_prev.at(targets[i]) * d_prev,
                sizeof(double) * d_prev);
}

// Algorithm 2, sampling part: S^(K) = M; S^(k-1) = S^(k) united with N(u) for
// every u in S^(k), with N given by `nbr_row`.
template <typename NbrRow>
std::vector<std::vector<int32_t>> minibatch_sets_impl(const int32_t* targets,
                                                      int64_t num_targets, int K, int T,
                                                      NbrRow nbr_row) {
  std::vector<std::set<int32_t>> Sset(K + 1);
  for (int64_t i = 0; i < num_targets; ++i) Sset[K].insert(targets[i]);
  for (int k = K; k >= 1; --k) {
    Sset[k - 1] = Sset[k];
    for (int32_t u : Sset[k]) {
      const int32_t* ids = nbr_row(u);
      for (int t = 0; t < T; ++t)
        if (ids[t] >= 0) Sset[k - 1].insert(ids[t]);
    }
  }
  std::vector<std::vector<int32_t>> S(K + 1);
  for (int k = 0; k <= K; ++k) S[k].assign(Sset[k].begin(), Sset[k].end());
  return S;
}

// Sampled Algorithm 2 state: the sets S^(0..K) and the neighbourhood rows of
// every node of S^(1) (which holds S^(2..K) too), each computed by the walks
// of Sec. 3.2 for that node alone.
struct Sample {
  std::vector<std::vector<int32_t>> S;
  std::vector<int32_t> rows_ids;  // sorted ids owning a neighbourhood row
  std::vector<int32_t> idx;
  std::vector<float> wts;
  int T = 0;
};

}  // namespace

extern "C" {

void orc_minibatch_embed(const int32_t* targets, int64_t num_targets, int K, const double* x,
                         int d0, const int32_t* nbr_idx, const float* nbr_w, int T,
                         const double* const* Qs, const double* const* qs, const int* ms,
                         const double* const* Ws, const double* const* ws, const int* d_outs,
                         double* out, int nthreads, const int* pools) {
  auto ids_of = [&](int32_t u) { return nbr_idx + (int64_t)u * T; };
  auto S = minibatch_sets_impl(targets, num_targets, K, T, ids_of);
  minibatch_embed_impl(
      targets, num_targets, K, S, [&](int32_t v) { return x + (int64_t)v * d0; }, d0,
      [&](int32_t u) {
        return std::make_pair(nbr_idx + (int64_t)u * T, nbr_w + (int64_t)u * T);
      },
      T, Qs, qs, ms, Ws, ws, d_outs, pools, out, nthreads);
}

// Sampling part of Algorithm 2 with neighbourhoods computed on demand, for
// graphs too large for an all-node table on the host. Returns a handle; read it
// with orc_sample_sizes / orc_sample_copy, release it with orc_sample_free.
void* orc_minibatch_sample(const int32_t* targets, int64_t num_targets, int K,
                           const int64_t* off, const int32_t* col, int64_t num_pins,
                           int64_t num_nodes, uint64_t seed, int walks, int hops, int T,
                           int nthreads) {
  Graph g{off, col, num_pins, num_nodes};
  Sample* smp = new Sample;
  smp->T = T;
  std::map<int32_t, int64_t> row_of;
  auto ensure_rows = [&](const std::vector<int32_t>& nodes) {
    std::vector<int32_t> todo;
    for (int32_t u : nodes)
      if (!row_of.count(u)) todo.push_back(u);
    const int64_t base = (int64_t)smp->rows_ids.size();
    smp->idx.resize((size_t)(base + (int64_t)todo.size()) * T);
    smp->wts.resize((size_t)(base + (int64_t)todo.size()) * T);
    std::vector<uint16_t> cnt((size_t)todo.size() * T);
    parallel_rows((int64_t)todo.size(), nthreads, [&](int64_t lo, int64_t hi) {
      std::vector<int32_t> visits;
      for (int64_t i = lo; i < hi; ++i) {
        visits.clear();
        walk_from(g, seed, todo[i], walks, hops, visits);
        select_top_t(visits, T, smp->idx.data() + (base + i) * T, cnt.data() + i * T,
                     smp->wts.data() + (base + i) * T);
      }
    });
    for (size_t i = 0; i < todo.size(); ++i) {
      row_of[todo[i]] = base + (int64_t)i;
      smp->rows_ids.push_back(todo[i]);
    }
  };
  // Expand level by level so that every node of S^(k), k >= 1, has its row.
  std::vector<std::set<int32_t>> Sset(K + 1);
  for (int64_t i = 0; i < num_targets; ++i) Sset[K].insert(targets[i]);
  for (int k = K; k >= 1; --k) {
    std::vector<int32_t> level(Sset[k].begin(), Sset[k].end());
    ensure_rows(level);
    Sset[k - 1] = Sset[k];
    for (int32_t u : level) {
      const int32_t* ids = smp->idx.data() + row_of.at(u) * T;
      for (int t = 0; t < T; ++t)
        if (ids[t] >= 0) Sset[k - 1].insert(ids[t]);
    }
  }
  smp->S.resize(K + 1);
  for (int k = 0; k <= K; ++k) smp->S[k].assign(Sset[k].begin(), Sset[k].end());
  // Store rows sorted by node id.
  std::vector<size_t> order(smp->rows_ids.size());
  for (size_t i = 0; i < order.size(); ++i) order[i] = i;
  std::sort(order.begin(), order.end(),
            [&](size_t a, size_t b) { return smp->rows_ids[a] < smp->rows_ids[b]; });
  std::vector<int32_t> ids2(order.size()), idx2(order.size() * T);
  std::vector<float> w2(order.size() * T);
  for (size_t i = 0; i < order.size(); ++i) {
    ids2[i] = smp->rows_ids[order[i]];
    std::memcpy(idx2.data() + i * T, smp->idx.data() + order[i] * T, sizeof(int32_t) * T);
    std::memcpy(w2.data() + i * T, smp->wts.data() + order[i] * T, sizeof(float) * T);
  }
  smp->rows_ids.swap(ids2);
  smp->idx.swap(idx2);
  smp->wts.swap(w2);
  return smp;
}

// sizes[0..K] = |S^(k)|, sizes[K+1] = number of neighbourhood rows.
void orc_sample_sizes(void* h, int K, int64_t* sizes) {
  Sample* smp = static_cast<Sample*>(h);
  for (int k = 0; k <= K; ++k) sizes[k] = (int64_t)smp->S[k].size();
  sizes[K + 1] = (int64_t)smp->rows_ids.size();
}

// sets: concatenated S^(0..K); row_ids, idx, wts: the neighbourhood rows.
void orc_sample_copy(void* h, int K, int32_t* sets, int32_t* row_ids, int32_t* idx, float* wts) {
  Sample* smp = static_cast<Sample*>(h);
  int64_t p = 0;
  for (int k = 0; k <= K; ++k)
    for (int32_t v : smp->S[k]) sets[p++] = v;
  std::memcpy(row_ids, smp->rows_ids.data(), sizeof(int32_t) * smp->rows_ids.size());
  std::memcpy(idx, smp->idx.data(), sizeof(int32_t) * smp->idx.size());
  std::memcpy(wts, smp->wts.data(), sizeof(float) * smp->wts.size());
}

void orc_sample_free(void* h) { delete static_cast<Sample*>(h); }

// Algorithm 2 embedding loop on a sample: x_ids (sorted) with their feature
// rows x_rows [n_x][d0] must cover S^(0); row_ids (sorted) with idx/wts
// [n_rows][T] must cover S^(1).
void orc_minibatch_embed_sampled(const int32_t* targets, int64_t num_targets, int K,
                                 const int32_t* x_ids, int64_t n_x, const double* x_rows, int d0,
                                 const int32_t* row_ids, int64_t n_rows, const int32_t* idx,
                                 const float* wts, int T, const double* const* Qs,
                                 const double* const* qs, const int* ms,
                                 const double* const* Ws, const double* const* ws,
                                 const int* d_outs, double* out, int nthreads,
                                 const int* pools) {
  auto find = [](const int32_t* ids, int64_t n, int32_t v) -> int64_t {
    const int32_t* p = std::lower_bound(ids, ids + n, v);
    return (p != ids + n && *p == v) ? (int64_t)(p - ids) : -1;
  };
  auto ids_of = [&](int32_t u) { return idx + find(row_ids, n_rows, u) * T; };
  auto S = minibatch_sets_impl(targets, num_targets, K, T, ids_of);
  minibatch_embed_impl(
      targets, num_targets, K, S,
      [&](int32_t v) { return x_rows + find(x_ids, n_x, v) * d0; }, d0,
      [&](int32_t u) {
        const int64_t r = find(row_ids, n_rows, u);
        return std::make_pair(idx + r * T, wts + r * T);
      },
      T, Qs, qs, ms, Ws, ws, d_outs, pools, out, nthreads);
}

// Algorithm 2, final loop: the output embedding z_u = G2 ReLU(G1 h_u + g) of
// each row, with G1 [d_hidden x d_in], g [d_hidden], G2 [d_out x d_hidden]
// (no bias and no activation after G2).
void orc_output_mlp(const double* h, int64_t n, int d_in, const double* G1, const double* g,
                    int d_hidden, const double* G2, int d_out, double* z, int nthreads) {
  parallel_rows(n, nthreads, [&](int64_t lo, int64_t hi) {
    std::vector<double> a((size_t)d_hidden);
    for (int64_t r = lo; r < hi; ++r) {
      for (int i = 0; i < d_hidden; ++i) {
        double acc = 0.0;
        for (int j = 0; j < d_in; ++j) acc += G1[(int64_t)i * d_in + j] * h[r * d_in + j];
        acc += g[i];
        a[i] = acc > 0.0 ? acc : 0.0;
      }
      for (int o = 0; o < d_out; ++o) {
        double acc = 0.0;
        for (int i = 0; i < d_hidden; ++i) acc += G2[(int64_t)o * d_hidden + i] * a[i];
        z[r * d_out + o] = acc;
      }
    }
  });
}

// Eq. (1), Sec. 3.3: for each pair (q, i), the expectation over negatives of
// max(0, z_q.z_n - z_q.z_i + margin). Readings: the expectation is the mean
// over the shared negative set, and the minibatch loss is the mean over pairs.
// Returns the minibatch loss; per_pair (nullable) receives each pair's term.
//
// With hard negatives (Sec. 3.3, "Hard negative items"): pair b also has its
// own items zhard[b][0..k) (entries with hard_valid[b][j] == 0 are absent),
// which join the negative set of that pair, so its term is the mean over the
// shared negatives and its present hard negatives together.
double orc_max_margin_loss_hard(const double* zq, const double* zpos, int64_t B,
                                const double* zneg, int64_t n_neg, const double* zhard,
                                const uint8_t* hard_valid, int64_t k, int d, double margin,
                                double* per_pair) {
  auto hinge = [&](int64_t b, const double* zn) {
    double pos = 0.0, neg = 0.0;
    for (int j = 0; j < d; ++j) pos += zq[b * d + j] * zpos[b * d + j];
    for (int j = 0; j < d; ++j) neg += zq[b * d + j] * zn[j];
    const double v = neg - pos + margin;
    return v > 0.0 ? v : 0.0;
  };
  double total = 0.0;
  for (int64_t b = 0; b < B; ++b) {
    double acc = 0.0;
    int64_t count = 0;
    for (int64_t n = 0; n < n_neg; ++n, ++count) acc += hinge(b, zneg + n * d);
    for (int64_t j = 0; j < k; ++j) {
      if (!hard_valid[b * k + j]) continue;
      acc += hinge(b, zhard + (b * k + j) * d);
      ++count;
    }
    const double term = count > 0 ? acc / (double)count : 0.0;
    if (per_pair) per_pair[b] = term;
    total += term;
  }
  return B > 0 ? total / (double)B : 0.0;
}

double orc_max_margin_loss(const double* zq, const double* zpos, int64_t B, const double* zneg,
                           int64_t n_neg, int d, double margin, double* per_pair) {
  return orc_max_margin_loss_hard(zq, zpos, B, zneg, n_neg, nullptr, nullptr, 0, d, margin,
                                  per_pair);
}

}  // extern "C"
