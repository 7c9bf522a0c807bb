// Offline catalog construction on the host (Sec. 4.1, Alg. 1).
//
// The catalog is enumerated slot by slot: every switch slot of a node picks
// the set of g outgoing lanes it launches (a combination of its candidate
// path instances), subject to resource disjointness (Eq. (1)/(4), tracked as
// one bit per directed resource) and the g-incoming limit per slot; a
// complete choice with every slot receiving exactly g lanes is a family.
// This visits exactly the compatible, complete instance sets that Alg. 1's
// include/exclude DFS reaches, each once: identical PIX copies are taken in
// copy order, which is PruneFamilies' exact-duplicate rule applied during the
// search.  PrunePaths runs before, the rest of PruneFamilies after.  With
// several NICs per switch, families that differ only by which of a
// switch's interchangeable NICs a lane uses are kept once (the smallest of
// each renaming class).
//
// Multi-node topologies use the node-circulant reduction: the same node-local
// pattern in every node, all NIC lanes of node n landing on node (n+k) mod
// n_nodes.  Shift 0 keeps NIC lanes inside the node (loopback through the two
// switches' NICs); shifts k != 0 use the NIC-carrying patterns, identical for
// every k.
#include <algorithm>
#include <cstring>
#include <map>
#include <set>
#include <exception>
#include <system_error>
#include <thread>
#include <tuple>

#include "internal.h"

namespace vp {
namespace {

struct Cand {
  int id, cls, src, dst, copy;
  int64_t bw;
  uint64_t res;   // bit per directed resource: UP q, DN q, TX (q, nic), RX (q, nic), socket link s -> s2
  bool remote;    // NIC lane to another node
};

struct Found {
  std::vector<int32_t> ids;   // ascending node-local ids
  std::vector<int32_t> L, R;  // Q x Q counts of intra-node / cross-node lanes
};

// Dominance between two path instances of one ordered pair (PrunePaths):
// no extra resource, no lower rate, and strictly better in one of the two.
bool path_dominates(const Cand& a, const Cand& b) {
  if (a.src != b.src || a.dst != b.dst || a.remote != b.remote) return false;
  bool subset = (a.res & ~b.res) == 0;
  if (!subset || a.bw < b.bw) return false;
  return a.res != b.res || a.bw > b.bw;
}

// fn(i) for every i in [0, n), on up to 16 host threads in contiguous
// blocks (the pruning rules judge each family or shape on its own).  A block
// whose thread cannot be started runs on the calling thread; an exception in
// any block is rethrown here after every thread has joined.
template <class Fn>
void parallel_for(size_t n, Fn fn) {
  const unsigned T = std::min<unsigned>(16, std::max(1u, std::thread::hardware_concurrency()));
  if (n < 4096 || T == 1) {
    for (size_t i = 0; i < n; ++i) fn(i);
    return;
  }
  const size_t chunk = (n + T - 1) / T;
  std::vector<std::exception_ptr> err(T);
  auto block = [&fn, &err, chunk, n](unsigned t) {
    try {
      for (size_t i = t * chunk; i < std::min(n, (t + 1) * chunk); ++i) fn(i);
    } catch (...) {
      err[t] = std::current_exception();
    }
  };
  std::vector<std::thread> th;
  for (unsigned t = 0; t < T; ++t) {
    try {
      th.emplace_back(block, t);
    } catch (const std::system_error&) {
      block(t);
    }
  }
  for (std::thread& x : th) x.join();
  for (const std::exception_ptr& e : err)
    if (e) std::rethrow_exception(e);
}

// Channel sets the search may record before the pruning rules run (a few
// GB of host memory at most): a node whose sets exceed it is refused rather
// than left to exhaust memory (eight switches of two GPUs already do).
constexpr size_t kMaxFound = size_t(1) << 22;

class SlotSearch {
 public:
  SlotSearch(const std::vector<Cand>& cands, int Q, int g) : Q_(Q), g_(g), out_(Q) {
    for (const Cand& c : cands) out_[c.src].push_back(c);
    indeg_.assign(Q, 0);
  }
  std::vector<Found> run() {
    slot(0, 0);
    return std::move(found_);
  }
  bool overflowed() const { return overflow_; }

 private:
  // choose g lanes for slot q, then recurse to slot q+1
  void slot(int q, uint64_t used) {
    if (overflow_) return;
    if (q == Q_) {
      for (int x = 0; x < Q_; ++x)
        if (indeg_[x] != g_) return;
      record();
      return;
    }
    pick(q, 0, 0, used);
  }
  void pick(int q, size_t from, int taken, uint64_t used) {
    if (taken == g_) {
      slot(q + 1, used);
      return;
    }
    const std::vector<Cand>& c = out_[q];
    for (size_t i = from; i + (size_t)(g_ - taken) <= c.size(); ++i) {
      const Cand& x = c[i];
      if (x.res & used) continue;
      if (indeg_[x.dst] >= g_) continue;
      // identical PIX copies enter in copy order only
      if (x.cls == VP_PATH_PIX && x.copy > 0) {
        bool prev = false;
        for (const Cand* y : chosen_)
          if (y->cls == VP_PATH_PIX && y->src == x.src && y->copy == x.copy - 1) prev = true;
        if (!prev) continue;
      }
      indeg_[x.dst]++;
      chosen_.push_back(&x);
      pick(q, i + 1, taken + 1, used | x.res);
      chosen_.pop_back();
      indeg_[x.dst]--;
    }
  }
  void record() {
    if (found_.size() >= kMaxFound) {
      overflow_ = true;
      return;
    }
    Found f;
    f.L.assign(Q_ * Q_, 0);
    f.R.assign(Q_ * Q_, 0);
    for (const Cand* c : chosen_) {
      f.ids.push_back(c->id);
      (c->remote ? f.R : f.L)[c->src * Q_ + c->dst]++;
    }
    std::sort(f.ids.begin(), f.ids.end());
    found_.push_back(std::move(f));
  }

  int Q_, g_;
  std::vector<std::vector<Cand>> out_;
  std::vector<int> indeg_;
  std::vector<const Cand*> chosen_;
  std::vector<Found> found_;
  bool overflow_ = false;
};

typedef std::tuple<int, int, bool, uint64_t> PairFoot;
typedef std::map<PairFoot, std::vector<int64_t>> Profile;

// Rates of a family's lanes per (pair, footprint), descending.
Profile profile_of(const Found& f, const std::vector<Cand>& by_id) {
  Profile m;
  for (int id : f.ids) {
    const Cand& c = by_id[id];
    m[PairFoot(c.src, c.dst, c.remote, c.res)].push_back(c.bw);
  }
  for (auto& kv : m) std::sort(kv.second.begin(), kv.second.end(), std::greater<int64_t>());
  return m;
}

// A lane's part of a family's profile as one word: the index of its (pair,
// footprint) among the table's distinct ones, then its rate.  A family's
// sorted words are its profile: two families have equal profiles exactly
// when they have the same multiset of (pair, footprint, rate).
std::vector<uint64_t> lane_words(const std::vector<Cand>& by_id) {
  std::map<PairFoot, uint64_t> foot;
  std::vector<uint64_t> w(by_id.size());
  for (const Cand& c : by_id) {
    auto it = foot.emplace(PairFoot(c.src, c.dst, c.remote, c.res), (uint64_t)foot.size()).first;
    w[c.id] = (it->second << 40) | (uint64_t)c.bw;   // rates are below 2^40 bytes/ns
  }
  return w;
}

uint64_t words_hash(const uint64_t* v, size_t n) {
  uint64_t h = 0x9E3779B97F4A7C15ull;
  for (size_t i = 0; i < n; ++i) {
    h ^= v[i] + 0x9E3779B97F4A7C15ull + (h << 6) + (h >> 2);
    h *= 0xFF51AFD7ED558CCDull;
  }
  return h ^ (h >> 32);
}

// Families sorted into canonical order, (L, R, ids) lexicographic: every
// family's three lists are written once as one flat big-endian 16-bit key
// (all values are below 2^16), and an index array is sorted by comparing
// keys as bytes.
void sort_canonical(std::vector<Found>& fs) {
  const size_t n = fs.size();
  if (n < 2) return;
  const size_t qq = fs[0].L.size(), w = fs[0].ids.size(), kl = 2 * (2 * qq + w);
  std::vector<uint8_t> key(n * kl);
  parallel_for(n, [&](size_t i) {
    uint8_t* k = key.data() + i * kl;
    auto put16 = [&](int v) {
      *k++ = (uint8_t)(v >> 8);
      *k++ = (uint8_t)v;
    };
    for (int v : fs[i].L) put16(v);
    for (int v : fs[i].R) put16(v);
    for (int v : fs[i].ids) put16(v);
  });
  std::vector<uint32_t> idx(n);
  for (size_t i = 0; i < n; ++i) idx[i] = (uint32_t)i;
  std::sort(idx.begin(), idx.end(), [&](uint32_t a, uint32_t b) {
    return std::memcmp(key.data() + a * kl, key.data() + b * kl, kl) < 0;
  });
  std::vector<Found> out(n);
  for (size_t i = 0; i < n; ++i) out[i] = std::move(fs[idx[i]]);
  fs.swap(out);
}

// PruneFamilies, first half: exact duplicates (same multiset of (pair,
// footprint, rate)) keep their first family in canonical order; the result
// is sorted by (L, R, ids), so every shape's families are contiguous.
// Profiles are compared through a 64-bit hash, every hash hit by the full
// sorted words.
std::vector<Found> drop_duplicates(std::vector<Found> fs, const std::vector<Cand>& by_id) {
  sort_canonical(fs);
  const std::vector<uint64_t> lw = lane_words(by_id);
  const size_t n = fs.size(), w = n ? fs[0].ids.size() : 0;
  std::vector<uint64_t> prof(n * w);
  // (hash, index) pairs sorted: equal profiles meet in one run of equal
  // hashes, where every family but the first of its profile is a duplicate
  std::vector<std::pair<uint64_t, uint32_t>> hi(n);
  parallel_for(n, [&](size_t i) {
    uint64_t* p = prof.data() + i * w;
    for (size_t x = 0; x < w; ++x) p[x] = lw[fs[i].ids[x]];
    std::sort(p, p + w);
    hi[i] = {words_hash(p, w), (uint32_t)i};
  });
  std::sort(hi.begin(), hi.end());
  std::vector<uint8_t> dup(n, 0);
  for (size_t b = 0, e; b < n; b = e) {
    for (e = b + 1; e < n && hi[e].first == hi[b].first; ++e) {
    }
    for (size_t x = b + 1; x < e; ++x)
      for (size_t y = b; y < x && !dup[hi[x].second]; ++y)
        if (!dup[hi[y].second] && std::equal(prof.data() + hi[x].second * w, prof.data() + (hi[x].second + 1) * w,
                                             prof.data() + hi[y].second * w))
          dup[hi[x].second] = 1;   // the run is in index order: y is the earlier family
  }
  std::vector<Found> uniq;
  for (size_t i = 0; i < n; ++i)
    if (!dup[i]) uniq.push_back(std::move(fs[i]));
  return uniq;
}

// PruneFamilies, second half: a family is dropped when another of its shape
// pairs with it per (pair, footprint) at no lower rate, one strictly higher.
// Shapes are contiguous in the input, so only families of one run compare.
std::vector<Found> drop_dominated(std::vector<Found> fs, const std::vector<Cand>& by_id) {
  const size_t n = fs.size();
  std::vector<Profile> prof(n);
  parallel_for(n, [&](size_t i) { prof[i] = profile_of(fs[i], by_id); });
  std::vector<size_t> runs;   // first family of every shape, then n
  for (size_t b = 0; b < n; ++b)
    if (b == 0 || fs[b].L != fs[b - 1].L || fs[b].R != fs[b - 1].R) runs.push_back(b);
  runs.push_back(n);
  std::vector<uint8_t> keep(n, 1);
  parallel_for(runs.size() - 1, [&](size_t r) {
    const size_t b = runs[r], e = runs[r + 1];
    for (size_t i = b; i < e; ++i) {
      bool dominated = false;
      for (size_t j = b; j < e && !dominated; ++j) {
        if (i == j || prof[i].size() != prof[j].size()) continue;
        bool ok = true, strict = false;
        for (auto it = prof[j].begin(); it != prof[j].end() && ok; ++it) {
          auto jt = prof[i].find(it->first);
          if (jt == prof[i].end() || jt->second.size() != it->second.size()) { ok = false; break; }
          for (size_t x = 0; x < it->second.size(); ++x) {
            if (it->second[x] < jt->second[x]) ok = false;
            if (it->second[x] > jt->second[x]) strict = true;
          }
        }
        dominated = ok && strict;
      }
      keep[i] = !dominated;
    }
  });
  std::vector<Found> out;
  for (size_t i = 0; i < n; ++i)
    if (keep[i]) out.push_back(std::move(fs[i]));
  return out;
}

}  // namespace

namespace {

// Families that differ only by which of a switch's interchangeable NICs
// each lane uses are one family: a family is kept when renaming the NICs of
// the slots (one permutation per slot, on the source NIC of the lanes it
// sends and the destination NIC of the lanes it receives) never yields a
// smaller ascending id list.  Every renaming of a slot's NICs is tried.
std::vector<Found> nic_representatives(std::vector<Found> fs, const std::vector<Cand>& by_id, int Q, int m) {
  if (m == 1) return fs;
  // id of each NIC instance by (src, dst, copy)
  std::map<std::tuple<int, int, int>, int> nic;
  for (const Cand& c : by_id)
    if (c.cls == VP_PATH_NIC) nic[std::make_tuple(c.src, c.dst, c.copy)] = c.id;
  std::vector<std::vector<int>> sym;   // the m! permutations of one slot's NICs
  std::vector<int> perm(m);
  for (int x = 0; x < m; ++x) perm[x] = x;
  do sym.push_back(perm); while (std::next_permutation(perm.begin(), perm.end()));
  int64_t combos = 1;
  for (int q = 0; q < Q; ++q) combos *= (int64_t)sym.size();
  std::vector<uint8_t> keep(fs.size());
  parallel_for(fs.size(), [&](size_t fi) {
    const Found& f = fs[fi];
    std::vector<int32_t> renamed;
    bool least = true;
    for (int64_t code = 1; code < combos && least; ++code) {
      renamed.clear();
      for (int32_t id : f.ids) {
        const Cand& c = by_id[id];
        if (c.cls != VP_PATH_NIC) {
          renamed.push_back(id);
          continue;
        }
        int64_t cs = code, cd = code;
        for (int q = 0; q < c.src; ++q) cs /= (int64_t)sym.size();
        for (int q = 0; q < c.dst; ++q) cd /= (int64_t)sym.size();
        const int x = sym[cs % (int64_t)sym.size()][c.copy / m], y = sym[cd % (int64_t)sym.size()][c.copy % m];
        renamed.push_back(nic.at(std::make_tuple(c.src, c.dst, x * m + y)));
      }
      std::sort(renamed.begin(), renamed.end());
      least = !(renamed < f.ids);
    }
    keep[fi] = least;
  });
  std::vector<Found> out;
  for (size_t fi = 0; fi < fs.size(); ++fi)
    if (keep[fi]) out.push_back(std::move(fs[fi]));
  return out;
}

}  // namespace

namespace {

// Node-local instance table in canonical id order: (class, src, dst, copy).
// A NIC instance leaves through NIC x of its source switch and arrives
// through NIC y of its destination switch (copy = x * m + y, m NICs per
// switch); every GPU of a switch reaches each of the switch's NICs.
std::vector<Cand> instance_table(const vp_topology& t) {
  const int W = t.switches_per_socket, g = t.gpus_per_switch;
  const int Q = t.sockets_per_node * W, m = t.nics_per_switch;
  const int64_t pcie = t.pcie_bytes_per_ns;
  const int64_t nicbw = std::min(t.pcie_bytes_per_ns, t.nic_bytes_per_ns);
  std::vector<Cand> table;
  const int S = t.sockets_per_node;
  auto bit = [](int r) { return (uint64_t)1 << r; };
  auto add = [&](int cls, int s, int d, int cp, int64_t bw, uint64_t res) {
    table.push_back(Cand{(int)table.size(), cls, s, d, cp, bw, res, false});
  };
  for (int q = 0; q < Q; ++q)
    for (int cp = 0; cp < g; ++cp) add(VP_PATH_PIX, q, q, cp, pcie, 0);
  for (int q = 0; q < Q; ++q)
    for (int q2 = 0; q2 < Q; ++q2)
      if (q != q2 && q / W == q2 / W) add(VP_PATH_PXB, q, q2, 0, pcie, bit(q) | bit(Q + q2));
  for (int q = 0; q < Q; ++q)
    for (int q2 = 0; q2 < Q; ++q2)
      for (int x = 0; x < m; ++x)
        for (int y = 0; y < m; ++y)
          add(VP_PATH_NIC, q, q2, x * m + y, nicbw, bit(2 * Q + q * m + x) | bit(2 * Q + Q * m + q2 * m + y));
  // peer to peer between sockets: both switches' root-complex links and the
  // directed link between the two sockets, at the PCIe rate
  if (t.flags & VP_TOPO_SYS_P2P)
    for (int q = 0; q < Q; ++q)
      for (int q2 = 0; q2 < Q; ++q2)
        if (q / W != q2 / W)
          add(VP_PATH_SYS, q, q2, 0, pcie, bit(q) | bit(Q + q2) | bit(2 * Q + 2 * Q * m + (q / W) * S + q2 / W));
  return table;
}

// PrunePaths over the table with NIC lanes local (remote = false) or to
// another node (remote = true): the instances that survive.
std::vector<Cand> prune_paths(const std::vector<Cand>& table, bool remote_nic) {
  std::vector<Cand> cand = table;
  for (Cand& x : cand) x.remote = remote_nic && x.cls == VP_PATH_NIC;
  std::vector<Cand> kept;
  for (const Cand& x : cand) {
    bool dom = false;
    for (const Cand& y : cand)
      if (y.id != x.id && path_dominates(y, x)) { dom = true; break; }
    if (!dom) kept.push_back(x);
  }
  return kept;
}

// Patterns (runs of families with one (L, R)) and the device image, from
// the canonical shift-0 and NIC-carrying family lists.
void fill_catalog(vp_catalog& c, const std::vector<Found>& f0, const std::vector<Found>& f1) {
  c.patL.clear(); c.patR.clear(); c.pat_fb.clear(); c.pat_fe.clear(); c.lfam.clear();
  auto group = [&](const std::vector<Found>& fs, int fam_base) {
    for (size_t i = 0; i < fs.size(); ++i) {
      if (i == 0 || fs[i].L != fs[i - 1].L || fs[i].R != fs[i - 1].R) {
        c.patL.push_back(fs[i].L);
        c.patR.push_back(fs[i].R);
        c.pat_fb.push_back(fam_base + (int)i);
        c.pat_fe.push_back(fam_base + (int)i);
      }
      c.pat_fe.back()++;
      c.lfam.push_back(fs[i].ids);
    }
  };
  group(f0, 0);
  c.J0 = (int)c.patL.size();
  c.F0 = (int)f0.size();
  group(f1, c.F0);
  c.J1 = (int)c.patL.size() - c.J0;
  c.F1 = (int)f1.size();
  build_device_image(c);
}

void set_shape(vp_catalog& c, const vp_topology& t) {
  c.topo = t;
  c.g = t.gpus_per_switch;
  c.Q = t.sockets_per_node * t.switches_per_socket;
  c.nn = t.n_nodes;
  c.G = c.nn * c.Q;
  c.N = c.G * c.g;
  const std::vector<Cand> table = instance_table(t);
  c.icls.clear(); c.isrc.clear(); c.idst.clear(); c.icopy.clear(); c.ibw.clear();
  for (const Cand& x : table) {
    c.icls.push_back(x.cls);
    c.isrc.push_back(x.src);
    c.idst.push_back(x.dst);
    c.icopy.push_back(x.copy);
    c.ibw.push_back(x.bw);
  }
}

// ------------------------------------------------------------ serialized form
//
// The compact serialized catalog (Table 4 sizes the catalog by such a
// payload) holds what Alg. 1 produced and nothing the topology alone gives:
//   magic "VPCATLG1" | topology: 6 x int32, 2 x int64 | F0, F1, Q*g: 3 x int32 |
//   (F0 + F1) x Q*g node-local instance ids (uint8, ascending per family) |
//   FNV-1a 64-bit hash of all preceding bytes.
// All integers little-endian.
constexpr char kMagic[8] = {'V', 'P', 'C', 'A', 'T', 'L', 'G', '1'};
constexpr size_t kHead = 8 + 6 * 4 + 2 * 8 + 3 * 4;

uint64_t fnv1a(const uint8_t* p, size_t n) {
  uint64_t h = 0xcbf29ce484222325ull;
  for (size_t i = 0; i < n; ++i) {
    h ^= p[i];
    h *= 0x100000001b3ull;
  }
  return h;
}

void put(std::vector<uint8_t>& b, uint64_t v, int bytes) {
  for (int i = 0; i < bytes; ++i) b.push_back((uint8_t)(v >> (8 * i)));
}

uint64_t get(const uint8_t* p, int bytes) {
  uint64_t v = 0;
  for (int i = 0; i < bytes; ++i) v |= (uint64_t)p[i] << (8 * i);
  return v;
}

}  // namespace

vp_status build_catalog_host(const vp_topology& t, vp_catalog& c) {
  set_shape(c, t);
  const std::vector<Cand> table = instance_table(t);
  bool overflow = false;
  auto enumerate = [&](bool remote_nic) {
    SlotSearch search(prune_paths(table, remote_nic), c.Q, c.g);
    std::vector<Found> raw = search.run();
    if (search.overflowed()) {
      overflow = true;
      return std::vector<Found>();
    }
    std::vector<Cand> cand = table;
    for (Cand& x : cand) x.remote = remote_nic && x.cls == VP_PATH_NIC;
    // renaming a slot's NICs preserves dominance both ways, so the NIC
    // classes may be reduced to their representatives before it is checked
    std::vector<Found> fs = drop_dominated(
        nic_representatives(drop_duplicates(std::move(raw), cand), cand, c.Q, t.nics_per_switch), cand);
    if (remote_nic) {
      std::vector<Found> with_nic;
      for (Found& f : fs) {
        int n = 0;
        for (int v : f.R) n += v;
        if (n > 0) with_nic.push_back(std::move(f));
      }
      fs.swap(with_nic);
    }
    return fs;   // sorted by (L, R, ids): canonical
  };
  std::vector<Found> f0 = enumerate(false);
  std::vector<Found> f1 = c.nn > 1 && !overflow ? enumerate(true) : std::vector<Found>();
  if (overflow)
    return set_error(VP_ERR_UNSUPPORTED, "a node with this many switches has more candidate channels than the "
                                         "catalog search holds (2^22 before pruning)");
  fill_catalog(c, f0, f1);
  return VP_OK;
}

// Restricted catalogs for the peer/path ablation (Sec. 6.3): rule 1 keeps the
// families in which every lane takes its group pair's nearest path (PIX in a
// switch, PXB between two switches of one socket, SYS between sockets when
// enabled, the NICs otherwise), i.e. drops every family with a NIC lane
// between two switches of one node that a PCIe peer-to-peer path also joins.
// Canonical order is kept, so the result is a catalog of the same topology.
vp_status restrict_catalog(const vp_catalog& in, int rule, vp_catalog& out) {
  if (rule != 1) return set_error(VP_ERR_INVALID_ARGUMENT, "unknown catalog restriction");
  set_shape(out, in.topo);
  const std::vector<Cand> table = instance_table(in.topo);
  const int Q = out.Q, W = in.topo.switches_per_socket;
  const bool sys = (in.topo.flags & VP_TOPO_SYS_P2P) != 0;
  std::vector<Found> lists[2];
  for (int f = 0; f < in.F0 + in.F1; ++f) {
    const bool remote = f >= in.F0;
    Found fam;
    fam.L.assign(Q * Q, 0);
    fam.R.assign(Q * Q, 0);
    bool keep = true;
    for (int id : in.lfam[f]) {
      const Cand& y = table[id];
      const bool nic = y.cls == VP_PATH_NIC;
      if (nic && !remote && y.src != y.dst && (sys || y.src / W == y.dst / W)) keep = false;
      ((nic && remote) ? fam.R : fam.L)[y.src * Q + y.dst]++;
      fam.ids.push_back(id);
    }
    if (keep) lists[remote ? 1 : 0].push_back(std::move(fam));
  }
  fill_catalog(out, lists[0], lists[1]);
  return VP_OK;
}

std::vector<uint8_t> serialize_catalog(const vp_catalog& c) {
  std::vector<uint8_t> b(kMagic, kMagic + 8);
  const vp_topology& t = c.topo;
  for (int32_t v : {t.n_nodes, t.sockets_per_node, t.switches_per_socket, t.gpus_per_switch, t.nics_per_switch,
                    t.flags})
    put(b, (uint32_t)v, 4);
  put(b, (uint64_t)t.pcie_bytes_per_ns, 8);
  put(b, (uint64_t)t.nic_bytes_per_ns, 8);
  put(b, (uint32_t)c.F0, 4);
  put(b, (uint32_t)c.F1, 4);
  put(b, (uint32_t)(c.Q * c.g), 4);
  for (const std::vector<int32_t>& f : c.lfam)
    for (int32_t id : f) b.push_back((uint8_t)id);
  put(b, fnv1a(b.data(), b.size()), 8);
  return b;
}

// Rebuilds a catalog from its serialized form.  Everything Alg. 1 guarantees
// is checked again: every family is a complete, resource-disjoint set of
// surviving path instances (Eq. (1), Eq. (4)), identical PIX copies appear in
// copy order, NIC-carrying families carry a NIC lane, every family is the
// representative of its NIC renaming class, and each list is in strictly
// increasing canonical order (no duplicates).  A subset of the
// families Alg. 1 would find is accepted (a restricted catalog).
vp_status deserialize_catalog(const uint8_t* p, size_t n, vp_catalog& c,
                              vp_status (*check_topology)(const vp_topology&)) {
  if (n < kHead + 8 || std::memcmp(p, kMagic, 8) != 0)
    return set_error(VP_ERR_INVALID_ARGUMENT, "not a serialized catalog");
  if (get(p + n - 8, 8) != fnv1a(p, n - 8)) return set_error(VP_ERR_INVALID_ARGUMENT, "catalog checksum mismatch");
  vp_topology t;
  const uint8_t* q = p + 8;
  t.n_nodes = (int32_t)get(q, 4); t.sockets_per_node = (int32_t)get(q + 4, 4);
  t.switches_per_socket = (int32_t)get(q + 8, 4); t.gpus_per_switch = (int32_t)get(q + 12, 4);
  t.nics_per_switch = (int32_t)get(q + 16, 4); t.flags = (int32_t)get(q + 20, 4);
  t.pcie_bytes_per_ns = (int64_t)get(q + 24, 8); t.nic_bytes_per_ns = (int64_t)get(q + 32, 8);
  q += 40;
  vp_status st = check_topology(t);
  if (st != VP_OK) return st;
  const int64_t F0 = (int32_t)get(q, 4), F1 = (int32_t)get(q + 4, 4), QG = (int32_t)get(q + 8, 4);
  q += 12;
  set_shape(c, t);
  const int Q = c.Q, g = c.g;
  if (QG != Q * g || F0 < 1 || F1 < 0 || (c.nn == 1) != (F1 == 0) ||
      (size_t)((F0 + F1) * QG) != n - kHead - 8)
    return set_error(VP_ERR_INVALID_ARGUMENT, "catalog sizes do not match its topology");
  const std::vector<Cand> table = instance_table(t);
  const int n_inst = (int)table.size();
  std::vector<Found> lists[2];
  for (int part = 0; part < 2; ++part) {
    const bool remote = part == 1;
    std::vector<char> kept(n_inst, 0);
    for (const Cand& x : prune_paths(table, remote)) kept[x.id] = 1;
    for (int64_t f = 0; f < (part ? F1 : F0); ++f) {
      Found fam;
      fam.L.assign(Q * Q, 0);
      fam.R.assign(Q * Q, 0);
      std::vector<int> outd(Q, 0), ind(Q, 0);
      uint64_t used = 0;
      bool ok = true;
      int nic = 0;
      for (int64_t x = 0; x < QG; ++x) {
        const int id = *q++;
        if (id >= n_inst || !kept[id] || (!fam.ids.empty() && id <= fam.ids.back())) { ok = false; continue; }
        const Cand& y = table[id];
        if (y.res & used) ok = false;
        used |= y.res;
        if (y.cls == VP_PATH_PIX && y.copy > 0 &&
            std::find(fam.ids.begin(), fam.ids.end(), id - 1) == fam.ids.end())
          ok = false;
        outd[y.src]++;
        ind[y.dst]++;
        const bool r = remote && y.cls == VP_PATH_NIC;
        nic += r;
        (r ? fam.R : fam.L)[y.src * Q + y.dst]++;
        fam.ids.push_back(id);
      }
      for (int s = 0; s < Q; ++s) ok = ok && outd[s] == g && ind[s] == g;
      if (remote && nic == 0) ok = false;
      if (!ok) return set_error(VP_ERR_INVALID_ARGUMENT, "serialized catalog holds an infeasible family");
      if (!lists[part].empty() && !(std::tie(lists[part].back().L, lists[part].back().R, lists[part].back().ids) <
                                   std::tie(fam.L, fam.R, fam.ids)))
        return set_error(VP_ERR_INVALID_ARGUMENT, "serialized families are not in canonical order");
      lists[part].push_back(std::move(fam));
    }
    // several NICs per switch: every family must be its renaming class's
    // representative
    std::vector<Cand> cand = table;
    for (Cand& x : cand) x.remote = remote && x.cls == VP_PATH_NIC;
    if (nic_representatives(lists[part], cand, Q, t.nics_per_switch).size() != lists[part].size())
      return set_error(VP_ERR_INVALID_ARGUMENT, "serialized catalog holds a family under other NIC names");
  }
  fill_catalog(c, lists[0], lists[1]);
  return VP_OK;
}

void build_device_image(vp_catalog& c) {
  DevCatalogLayout& L = c.lay;
  const int Q = c.Q, g = c.g, QG = Q * g, P = c.J0 + c.J1, FL = c.F0 + c.F1;
  L.N = c.N; L.G = c.G; L.g = g; L.Q = Q; L.nn = c.nn; L.n_inst = (int)c.icls.size();
  L.J0 = c.J0; L.J1 = c.J1; L.F0 = c.F0; L.F1 = c.F1;
  L.J = (int64_t)c.J0 + (int64_t)c.J1 * (c.nn - 1);
  L.F = (int64_t)c.F0 + (int64_t)c.F1 * (c.nn - 1);
  int ts = 1;
  for (int p = 0; p < P; ++p) {
    int n = 0;
    for (int x = 0; x < Q * Q; ++x) n += (c.patL[p][x] != 0) + (c.patR[p][x] != 0);
    ts = std::max(ts, n);
  }
  L.TS = ts;
  int np = 1;
  for (int x = 2; x <= g; ++x) np *= x;
  L.n_perm = np;
  int off = 0;
  L.off_terms = off; off += P * ts;
  L.off_nterms = off; off += P;
  L.off_fb = off; off += P;
  L.off_fe = off; off += P;
  L.off_fam_info = off; off += FL * QG;
  L.off_fam_out = off; off += FL * QG;
  L.off_fam_in = off; off += FL * QG;
  L.off_perms = off; off += np * g;
  // distinct NIC-lane sets of the NIC-carrying patterns: the shift part of a
  // shape's score depends on its pattern only through this set
  std::map<std::vector<int>, int> set_id;
  std::vector<std::vector<int>> sets;
  std::vector<int> psid(c.J1);
  for (int p = c.J0; p < P; ++p) {
    std::vector<int> e;   // a slot pair appears once per NIC lane on it
    for (int x = 0; x < Q * Q; ++x)
      for (int r = 0; r < c.patR[p][x]; ++r) e.push_back(x);
    auto it = set_id.find(e);
    if (it == set_id.end()) {
      it = set_id.emplace(e, (int)sets.size()).first;
      sets.push_back(e);
    }
    psid[p - c.J0] = it->second;
  }
  L.nS = (int)sets.size();
  L.off_rset = off; off += L.nS * kMaxRTerms;
  L.off_psid = off; off += c.J1;
  L.total = off;
  // every path but NIC runs at the PCIe rate; the planner relies on it (one
  // largest-lane maximum for the PCIe-rate classes, one for NIC)
  L.bw_cls[VP_PATH_PIX] = c.topo.pcie_bytes_per_ns;
  L.bw_cls[VP_PATH_PXB] = c.topo.pcie_bytes_per_ns;
  L.bw_cls[VP_PATH_NIC] = std::min(c.topo.pcie_bytes_per_ns, c.topo.nic_bytes_per_ns);
  L.bw_cls[VP_PATH_SYS] = c.topo.pcie_bytes_per_ns;
  L.bw_max = std::max(L.bw_cls[0], L.bw_cls[2]);

  std::vector<int32_t>& im = c.image;
  im.assign(off, 0);
  for (int p = 0; p < P; ++p) {
    int n = 0;
    for (int block = 0; block < 2; ++block)
      for (int q = 0; q < Q; ++q)
        for (int q2 = 0; q2 < Q; ++q2) {
          int cnt = (block ? c.patR[p] : c.patL[p])[q * Q + q2];
          if (cnt) im[L.off_terms + p * ts + n++] = cnt | (q2 << 4) | (q << 8) | (block << 12);
        }
    im[L.off_nterms + p] = n;
    im[L.off_fb + p] = c.pat_fb[p];
    im[L.off_fe + p] = c.pat_fe[p];
  }
  for (int f = 0; f < FL; ++f) {
    std::vector<int> no(Q, 0), ni(Q, 0);
    for (int x = 0; x < QG; ++x) {
      int id = c.lfam[f][x];
      im[L.off_fam_info + f * QG + x] = c.icls[id] | (c.isrc[id] << 4) | (c.idst[id] << 8) | (id << 12);
      im[L.off_fam_out + f * QG + c.isrc[id] * g + no[c.isrc[id]]++] = x;
      im[L.off_fam_in + f * QG + c.idst[id] * g + ni[c.idst[id]]++] = x;
    }
  }
  for (int si = 0; si < L.nS; ++si)
    for (int m = 0; m < kMaxRTerms; ++m)
      im[L.off_rset + si * kMaxRTerms + m] = m < (int)sets[si].size() ? sets[si][m] : -1;
  for (int p = 0; p < c.J1; ++p) im[L.off_psid + p] = psid[p];
  std::vector<int> perm(g);
  for (int x = 0; x < g; ++x) perm[x] = x;
  int pi = 0;
  do {
    for (int x = 0; x < g; ++x) im[L.off_perms + pi * g + x] = perm[x];
    ++pi;
  } while (std::next_permutation(perm.begin(), perm.end()));
}

}  // namespace vp
