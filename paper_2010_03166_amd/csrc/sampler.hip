// Frontier sampling of minibatch node sets on the host (Section 4.1,
// Algorithm 2) with the Dashboard of Section 4.2 (Algorithms 3 and 4), and
// the pool of Section 6.3 (Algorithm 8) that keeps several subgraphs sampled
// ahead of the GPU by worker threads.  Host code only: the GPU receives each
// node list and induces the subgraph itself (induce.hip).
//
// Dashboard.  Every frontier node v owns a tile (its node id and the range
// of its pins) and deg(v) consecutive pins in DB, each naming the tile;
// probing DB uniformly until a pin is hit therefore picks a frontier node
// with probability proportional to its degree.  Popping a node clears its
// pins, adding one appends pins at the end; when the end is reached the
// live tiles are compacted to the front (cleanup).  A node whose degree
// exceeds the free slots even after a cleanup gets the free slots only.
//
// Random numbers: SplitMix64 (Steele, Lea, Flood, OOPSLA 2014), used as a
// counter-based generator: the k-th output of a generator started at state
// s is mix(s + (k+1) * 0x9E3779B97F4A7C15).  Subgraph `id` draws from four
// streams whose start states are outputs 4*id + purpose of the generator
// started at the seed (0 initial frontier, 1 probes, 2 neighbour choice,
// 3 clipping); an integer below k is floor(r * k / 2^64).  Probes are drawn
// one after another from stream 1 until one hits a pin, so the outcome does
// not depend on how many probes are tried at once.
#include <algorithm>
#include <cmath>
#include <condition_variable>
#include <map>
#include <mutex>
#include <new>
#include <thread>
#include <unordered_set>
#include <vector>

#include "abi.hpp"

using namespace gnnprop;

namespace {

constexpr uint64_t GOLDEN = 0x9E3779B97F4A7C15ull;

inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// k-th output of a SplitMix64 generator started at `state`
inline uint64_t splitmix(uint64_t state, uint64_t k) { return mix64(state + (k + 1) * GOLDEN); }

inline uint64_t below(uint64_t r, uint64_t k) {
  return (uint64_t)(((unsigned __int128)r * (unsigned __int128)k) >> 64);
}

struct Stream {
  uint64_t state, count = 0;
  Stream(uint64_t seed, int64_t id, int purpose)
      : state(splitmix(seed, 4 * (uint64_t)id + (uint64_t)purpose)) {}
  uint64_t next() { return splitmix(state, count++); }
};

struct FullGraph {
  int64_t n;
  const int64_t* indptr;
  const int32_t* indices;
};

struct Params {
  int32_t m, budget, clip;
  double eta;
};

// The Dashboard (DB) and its index array (IA: a tile's first pin, its node
// and whether it is in the frontier).
class Dashboard {
 public:
  explicit Dashboard(int64_t cap) : db_(cap, -1) {}
  int64_t cap() const { return (int64_t)db_.size(); }
  int64_t valid() const { return valid_; }
  int64_t free_slots() const { return cap() - used_; }

  void add(int32_t v, int64_t pins) {
    const int32_t t = (int32_t)node_.size();
    node_.push_back(v);
    first_.push_back(used_);
    pins_.push_back(pins);
    live_.push_back(1);
    std::fill(db_.begin() + used_, db_.begin() + used_ + pins, t);
    used_ += pins;
    valid_ += pins;
  }

  // Probe until a pin is hit; clears the hit node's pins; returns its node.
  int32_t pop(Stream& probes) {
    int32_t t;
    do {
      t = db_[below(probes.next(), (uint64_t)cap())];
    } while (t < 0);
    std::fill(db_.begin() + first_[t], db_.begin() + first_[t] + pins_[t], -1);
    valid_ -= pins_[t];
    live_[t] = 0;
    return node_[t];
  }

  // Moves the live tiles' pins to the front, in tile order.
  void cleanup() {
    std::vector<int32_t> node;
    std::vector<int64_t> first, pins;
    int64_t pos = 0;
    std::fill(db_.begin(), db_.end(), -1);
    for (size_t t = 0; t < node_.size(); ++t) {
      if (!live_[t]) continue;
      const int32_t nt = (int32_t)node.size();
      std::fill(db_.begin() + pos, db_.begin() + pos + pins_[t], nt);
      node.push_back(node_[t]);
      first.push_back(pos);
      pins.push_back(pins_[t]);
      pos += pins_[t];
    }
    node_.swap(node);
    first_.swap(first);
    pins_.swap(pins);
    live_.assign(node_.size(), 1);
    used_ = pos;
  }

 private:
  std::vector<int32_t> db_;
  std::vector<int32_t> node_;
  std::vector<int64_t> first_, pins_;
  std::vector<uint8_t> live_;
  int64_t used_ = 0, valid_ = 0;
};

inline int64_t degree(const FullGraph& g, int32_t v) { return g.indptr[v + 1] - g.indptr[v]; }

// One subgraph's node set, sorted.
void frontier_sample(const FullGraph& g, const Params& p, uint64_t seed, int64_t id,
                     std::vector<int32_t>& out) {
  out.clear();
  if (g.n == 0) return;
  Stream s_init(seed, id, 0), s_probe(seed, id, 1), s_nbr(seed, id, 2), s_clip(seed, id, 3);
  const double d = (double)g.indptr[g.n] / (double)g.n;
  const int64_t cap = std::max<int64_t>(1, (int64_t)std::ceil(p.eta * p.m * d));
  Dashboard db(cap);
  // the initial frontier: m distinct nodes, uniformly
  const int64_t m = std::min<int64_t>(p.m, g.n);
  std::vector<int32_t> fs;
  std::unordered_set<int32_t> chosen;
  while ((int64_t)fs.size() < m) {
    const int32_t u = (int32_t)below(s_init.next(), (uint64_t)g.n);
    if (chosen.insert(u).second) fs.push_back(u);
  }
  for (int32_t v : fs) db.add(v, std::min(degree(g, v), db.free_slots()));
  out = fs;  // V_s starts as the initial frontier
  for (int64_t it = 0; it < (int64_t)p.budget - m; ++it) {
    if (db.valid() == 0) break;  // no frontier node has a pin left
    const int32_t v_pop = db.pop(s_probe);
    const int64_t dp = degree(g, v_pop);
    const int32_t v_new = g.indices[g.indptr[v_pop] + (int64_t)below(s_nbr.next(), (uint64_t)dp)];
    int64_t k = degree(g, v_new);
    if (k > db.free_slots()) db.cleanup();
    k = std::min(k, db.free_slots());
    db.add(v_new, k);
    out.push_back(v_new);  // V_s gains the node entering the frontier
  }
  std::sort(out.begin(), out.end());
  out.erase(std::unique(out.begin(), out.end()), out.end());
  // clipping (Section 6.2): drop |V_s| mod clip nodes chosen uniformly
  if (p.clip > 1) {
    const size_t drop = out.size() % (size_t)p.clip;
    for (size_t r = 0; r < drop; ++r)
      out.erase(out.begin() + (ptrdiff_t)below(s_clip.next(), out.size()));
  }
}

gnn_status check_params(int64_t n_full, const int64_t* indptr, const int32_t* indices,
                        int32_t m, int32_t budget, double eta, int32_t clip) {
  if (n_full < 0 || n_full > INT32_MAX || m < 1 || budget < m || clip < 0 ||
      !(eta >= 1.0) || !std::isfinite(eta))
    return GNN_ERR_SHAPE;
  if (n_full > 0 && (!indptr || (indptr[n_full] > 0 && !indices))) return GNN_ERR_NULL;
  return GNN_OK;
}

}  // namespace

struct gnn_sampler {
  FullGraph g;
  Params p;
  uint64_t seed;
  int32_t depth;
  std::vector<std::thread> workers;
  std::mutex mu;
  std::condition_variable ready, space;
  int64_t next_sample = 0, next_pop = 0;
  std::map<int64_t, std::vector<int32_t>> done;
  bool stop = false, failed = false;

  void work() {
    std::vector<int32_t> nodes;
    for (;;) {
      int64_t id;
      {
        std::unique_lock<std::mutex> lk(mu);
        space.wait(lk, [&] { return stop || next_sample - next_pop < depth; });
        if (stop) return;
        id = next_sample++;
      }
      bool ok = true;
      try {
        frontier_sample(g, p, seed, id, nodes);
      } catch (...) {
        ok = false;
      }
      std::lock_guard<std::mutex> lk(mu);
      if (!ok) failed = true;
      done[id] = nodes;
      ready.notify_all();
    }
  }
};

extern "C" {

gnn_status gnn_frontier_sample(int64_t n_full, const int64_t* indptr,
                               const int32_t* indices, int32_t m, int32_t budget,
                               double eta, int32_t clip, uint64_t seed, int64_t id,
                               int32_t* nodes, int32_t* n_nodes) {
  const gnn_status st = check_params(n_full, indptr, indices, m, budget, eta, clip);
  if (st != GNN_OK) return st;
  if (!nodes || !n_nodes) return GNN_ERR_NULL;
  std::vector<int32_t> out;
  try {
    frontier_sample(FullGraph{n_full, indptr, indices}, Params{m, budget, clip, eta}, seed, id,
                    out);
  } catch (...) {
    return GNN_ERR_HIP;
  }
  std::copy(out.begin(), out.end(), nodes);
  *n_nodes = (int32_t)out.size();
  return GNN_OK;
}

gnn_status gnn_sampler_create(int64_t n_full, const int64_t* indptr,
                              const int32_t* indices, int32_t m, int32_t budget,
                              double eta, int32_t clip, uint64_t seed,
                              int32_t threads, int32_t depth, gnn_sampler** out) {
  const gnn_status st = check_params(n_full, indptr, indices, m, budget, eta, clip);
  if (st != GNN_OK) return st;
  if (!out) return GNN_ERR_NULL;
  if (threads < 1 || depth < 1) return GNN_ERR_SHAPE;
  gnn_sampler* s = new (std::nothrow) gnn_sampler;
  if (!s) return GNN_ERR_HIP;
  s->g = FullGraph{n_full, indptr, indices};
  s->p = Params{m, budget, clip, eta};
  s->seed = seed;
  s->depth = depth;
  try {
    for (int32_t t = 0; t < threads; ++t) s->workers.emplace_back([s] { s->work(); });
  } catch (...) {
    {
      std::lock_guard<std::mutex> lk(s->mu);
      s->stop = true;
    }
    s->space.notify_all();
    for (auto& w : s->workers) w.join();
    delete s;
    return GNN_ERR_HIP;
  }
  *out = s;
  return GNN_OK;
}

gnn_status gnn_sampler_next(gnn_sampler* s, int32_t* nodes, int32_t* n_nodes, int64_t* id) {
  if (!s || !nodes || !n_nodes) return GNN_ERR_NULL;
  std::vector<int32_t> v;
  int64_t k;
  {
    std::unique_lock<std::mutex> lk(s->mu);
    k = s->next_pop;
    s->ready.wait(lk, [&] { return s->done.count(k) > 0; });
    if (s->failed) return GNN_ERR_HIP;
    v.swap(s->done[k]);
    s->done.erase(k);
    s->next_pop++;
  }
  s->space.notify_all();
  std::copy(v.begin(), v.end(), nodes);
  *n_nodes = (int32_t)v.size();
  if (id) *id = k;
  return GNN_OK;
}

void gnn_sampler_destroy(gnn_sampler* s) {
  if (!s) return;
  {
    std::lock_guard<std::mutex> lk(s->mu);
    s->stop = true;
  }
  s->space.notify_all();
  for (auto& w : s->workers) w.join();
  delete s;
}

}  // extern "C"
