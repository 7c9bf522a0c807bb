// ORACLE -- TEST INFRASTRUCTURE ONLY.
//
// A plain, slow, single-threaded CPU implementation of the demand -> plan ->
// pack path of VarioPath (arxiv 2609.34340), written from the paper, and of
// the receive side and the combine direction that the same buffer layout
// implies (unpack into the expert-major output; combine pack and unpack on a
// schedule planned for the transposed demand).  Only the
// tests, the smoke check and the benchmark's CPU-baseline leg may load it.  It
// shares no code, header, table or helper with the HIP library; the two meet
// only at the seeded inputs.  Every function names the passage it follows.
//
// Where the paper fixes a result by a plain definition (the demand matrix,
// the send-buffer layout, the modeled completion time) the code is that
// definition written out.  So is the catalog: every set of path instances
// that satisfies the balance and compatibility constraints (Eq. (3),
// Eq. (4)), found by a search over each group's choice of outgoing lanes,
// then pruned by the dominance rules of Sec. 4.1.  The scheduler is a
// heuristic: it takes the steps of Sec. 4.2 in the paper's order (shape by
// Eq. (5)-(6), binding by MultiStartAA on Eq. (7)-(8), volumes and utility
// by Eq. (9)-(10)), with every choice the paper leaves open fixed by the
// readings listed in the design notes (topology model, PIX multiplicity,
// node-circulant reduction, canonical order, integer credit, start rule,
// counter-based randomness, exact utility comparison).
//
// Arithmetic: int64 bytes and nanoseconds; utilities are compared exactly by
// cross-multiplication in unsigned 128-bit.  No floating point on the path.

#include <algorithm>
#include <cstdint>
#include <cstring>
#include <functional>
#include <map>
#include <set>
#include <tuple>
#include <vector>

namespace {

typedef int64_t i64;
typedef unsigned __int128 u128;

enum Status { OK = 0, INVALID_ARGUMENT = 1, INVALID_DEMAND = 2, NO_PROGRESS = 3,
              CAPACITY = 4, UNSUPPORTED = 5 };
enum Cls { PIX = 0, PXB = 1, NIC = 2, SYS = 3 };

struct Topo {
  int n_nodes, sockets, switches, g, nics;
  i64 pcie, nic;
  bool sys;   // GPUs under different sockets of a node reach each other peer to peer
  int Q() const { return sockets * switches; }        // switch slots per node
  int G() const { return n_nodes * Q(); }              // rank groups (one per switch)
  int N() const { return G() * g; }                    // ranks
};

// ---------------------------------------------------------------------------
// Group-level path instances (Sec. 4.1 "Topology abstraction"; Sec. 3 model
// setup).  Directed resources: per switch x, the uplink UP_x and downlink DN_x
// between the switch and its root complex; per NIC, TX and RX.  GPU<->switch
// links are endpoint-local and not modeled.  Path classes: PIX (same switch,
// no shared resource), PXB (same socket, other switch: UP_src, DN_dst) and NIC
// (any pair through one NIC of the source switch and one NIC of the
// destination switch: TX of the first, RX of the second; every GPU of a switch
// reaches every NIC of that switch inside the switch, so a switch with m NICs
// offers m x m NIC instances to each switch, `copy` = source NIC * m +
// destination NIC).  A path's rate is the minimum of its links.  With
// cross-socket peer-to-peer enabled, SYS joins two switches of different
// sockets of one node through both root complexes and the directed
// inter-socket link: UP_src, X(socket_src -> socket_dst), DN_dst, at the PCIe
// rate (the inter-socket link is taken to be faster than one PCIe link).
// ---------------------------------------------------------------------------
struct Inst {
  int id;          // canonical id (order of (cls, src, dst, copy))
  int cls;
  int a, d;        // source / destination group (slot for node-local sets)
  int copy;
  bool remote;     // NIC lane to another node (node-circulant sets only)
  i64 bw;
  std::vector<int> L;   // sorted resource ids
};

i64 rate_of(const Topo& t, int cls) {
  return cls == NIC ? std::min(t.pcie, t.nic) : t.pcie;
}

// Node-local instance table shared by the k = 0 (intra-node) and k != 0
// (remote) sets: PIX copies, PXB, and NIC for every slot pair and NIC pair.
// Resource ids: UP q -> q, DN q -> Q+q, TX of NIC x of slot q -> 2Q+q*m+x,
// RX of NIC y of slot q -> 2Q+Q*m+q*m+y, socket links after them.
std::vector<Inst> local_table(const Topo& t) {
  const int Q = t.Q();
  std::vector<Inst> v;
  for (int q = 0; q < Q; ++q)
    for (int c = 0; c < t.g; ++c)
      v.push_back({0, PIX, q, q, c, false, rate_of(t, PIX), {}});
  for (int q = 0; q < Q; ++q)
    for (int q2 = 0; q2 < Q; ++q2)
      if (q != q2 && q / t.switches == q2 / t.switches)
        v.push_back({0, PXB, q, q2, 0, false, rate_of(t, PXB), {q, Q + q2}});
  const int m = t.nics, X = 2 * Q + 2 * Q * m;   // socket links from X on
  for (int q = 0; q < Q; ++q)
    for (int q2 = 0; q2 < Q; ++q2)
      for (int x = 0; x < m; ++x)
        for (int y = 0; y < m; ++y)
          v.push_back({0, NIC, q, q2, x * m + y, false, rate_of(t, NIC),
                       {2 * Q + q * m + x, 2 * Q + Q * m + q2 * m + y}});
  // socket link s -> s2: resource X + s * sockets + s2
  if (t.sys)
    for (int q = 0; q < Q; ++q)
      for (int q2 = 0; q2 < Q; ++q2) {
        const int s = q / t.switches, s2 = q2 / t.switches;
        if (s != s2) v.push_back({0, SYS, q, q2, 0, false, rate_of(t, SYS), {q, Q + q2, X + s * t.sockets + s2}});
      }
  std::sort(v.begin(), v.end(), [](const Inst& x, const Inst& y) {
    return std::make_tuple(x.cls, x.a, x.d, x.copy) < std::make_tuple(y.cls, y.a, y.d, y.copy);
  });
  for (size_t i = 0; i < v.size(); ++i) v[i].id = (int)i;
  return v;
}

// Cluster-level instance set over all G groups (used for the full, unreduced
// Alg. 1 catalog of small topologies).  Resource ids: UP a -> a, DN a -> G+a,
// TX of NIC x of group a -> 2G+a*m+x, RX of NIC y of group d -> 2G+G*m+d*m+y,
// socket links after them.
std::vector<Inst> cluster_table(const Topo& t) {
  const int G = t.G(), Q = t.Q();
  std::vector<Inst> v;
  for (int a = 0; a < G; ++a)
    for (int c = 0; c < t.g; ++c)
      v.push_back({0, PIX, a, a, c, false, rate_of(t, PIX), {}});
  for (int a = 0; a < G; ++a)
    for (int d = 0; d < G; ++d) {
      bool same_node = a / Q == d / Q;
      bool same_socket = same_node && (a % Q) / t.switches == (d % Q) / t.switches;
      if (a != d && same_socket)
        v.push_back({0, PXB, a, d, 0, false, rate_of(t, PXB), {a, G + d}});
    }
  const int m = t.nics, X = 2 * G + 2 * G * m;
  for (int a = 0; a < G; ++a)
    for (int d = 0; d < G; ++d)
      for (int x = 0; x < m; ++x)
        for (int y = 0; y < m; ++y)
          v.push_back({0, NIC, a, d, x * m + y, false, rate_of(t, NIC),
                       {2 * G + a * m + x, 2 * G + G * m + d * m + y}});
  // socket link of node n, s -> s2: resource X + (n * sockets + s) * sockets + s2
  if (t.sys)
    for (int a = 0; a < G; ++a)
      for (int d = 0; d < G; ++d) {
        const int n = a / Q, s = (a % Q) / t.switches, s2 = (d % Q) / t.switches;
        if (n == d / Q && s != s2)
          v.push_back({0, SYS, a, d, 0, false, rate_of(t, SYS), {a, G + d, X + (n * t.sockets + s) * t.sockets + s2}});
      }
  std::sort(v.begin(), v.end(), [](const Inst& x, const Inst& y) {
    return std::make_tuple(x.cls, x.a, x.d, x.copy) < std::make_tuple(y.cls, y.a, y.d, y.copy);
  });
  for (size_t i = 0; i < v.size(); ++i) v[i].id = (int)i;
  return v;
}

bool subset_of(const std::vector<int>& x, const std::vector<int>& y) {
  return std::includes(y.begin(), y.end(), x.begin(), x.end());
}

// Path-level dominance (Sec. 4.1 "Pruning and search cost"): an instance is
// dropped when another instance of the same ordered group pair uses a subset
// of its resources at no lower rate, strictly better in one of the two.
std::vector<Inst> drop_dominated_paths(const std::vector<Inst>& R) {
  std::vector<Inst> out;
  for (const Inst& r : R) {
    bool dominated = false;
    for (const Inst& q : R) {
      if (&q == &r || q.a != r.a || q.d != r.d || q.remote != r.remote) continue;
      const bool fewer = subset_of(q.L, r.L) && q.L.size() < r.L.size();
      const bool faster = q.bw > r.bw;
      if (subset_of(q.L, r.L) && q.bw >= r.bw && (fewer || faster)) {
        dominated = true;
        break;
      }
    }
    if (!dominated) out.push_back(r);
  }
  return out;
}

// A family as the canonical ids of its instances (ascending).
typedef std::vector<int> Fam;

// Shape of a family: lane counts per (src group, dst group, remote flag).
typedef std::vector<int> ShapeKey;

// Every family of an instance set, from its definition (Sec. 4.1, Eq. (3)
// and Eq. (4)): a set of instances in which each group is the destination of
// exactly g instances and the source of exactly g, and no modeled resource
// is used twice.  The search decides one group at a time which g of the
// instances arriving at it the family takes (every g-subset, in index
// order); a choice is abandoned as soon as some group would send more than
// g lanes or a resource would repeat, and a complete choice is kept when
// every group sends exactly g.  The set of families found does not depend
// on the order of the search.
std::vector<std::vector<int>> all_families(const std::vector<Inst>& R, int n_groups, int g, int n_res) {
  std::vector<std::vector<int>> arriving(n_groups);
  for (int i = 0; i < (int)R.size(); ++i) arriving[R[i].d].push_back(i);
  std::vector<std::vector<int>> found;
  std::vector<int> sends(n_groups, 0), res_used(n_res, 0), chosen;

  auto fits = [&](int i) {
    if (sends[R[i].a] == g) return false;
    for (int l : R[i].L)
      if (res_used[l]) return false;
    return true;
  };
  auto take = [&](int i, int sgn) {
    sends[R[i].a] += sgn;
    for (int l : R[i].L) res_used[l] += sgn;
  };
  // group d picks its remaining `need` lanes among arriving[d][from..]
  std::function<void(int, int, int)> pick = [&](int d, int from, int need) {
    if (need == 0) {
      if (d + 1 < n_groups) {
        pick(d + 1, 0, g);
        return;
      }
      for (int x = 0; x < n_groups; ++x)
        if (sends[x] != g) return;
      found.push_back(chosen);
      return;
    }
    const std::vector<int>& opts = arriving[d];
    for (int k = from; k + need <= (int)opts.size(); ++k) {
      const int i = opts[k];
      if (!fits(i)) continue;
      take(i, +1);
      chosen.push_back(i);
      pick(d, k + 1, need - 1);
      chosen.pop_back();
      take(i, -1);
    }
  };
  if (n_groups > 0) pick(0, 0, g);
  return found;
}

// NIC symmetry (reading: the m NICs of a switch are interchangeable, same
// rate and same attachment): two families that differ only by a renaming of
// each group's NICs are one family under two names.  A family is kept only
// when no renaming (a permutation of the NICs of every group, applied to the
// source NIC of its lanes out of that group and to the destination NIC of
// its lanes into it) gives a smaller sorted id list.
std::vector<Fam> keep_nic_canonical(const std::vector<Fam>& fams, const std::vector<Inst>& table, int n_groups,
                                    int m) {
  if (m <= 1) return fams;
  std::map<std::tuple<int, int, int>, int> nic_id;   // (src group, dst group, copy) -> id
  for (const Inst& r : table)
    if (r.cls == NIC) nic_id[std::make_tuple(r.a, r.d, r.copy)] = r.id;
  std::vector<std::vector<int>> perms;
  std::vector<int> p(m);
  for (int x = 0; x < m; ++x) p[x] = x;
  do perms.push_back(p); while (std::next_permutation(p.begin(), p.end()));
  std::vector<Fam> out;
  for (const Fam& f : fams) {
    bool smallest = true;
    std::vector<int> pick(n_groups, 0);   // permutation index per group, odometer order
    while (smallest) {
      Fam img;
      for (int id : f) {
        const Inst& r = table[id];
        if (r.cls != NIC) {
          img.push_back(id);
          continue;
        }
        const int x = perms[pick[r.a]][r.copy / m], y = perms[pick[r.d]][r.copy % m];
        img.push_back(nic_id.at(std::make_tuple(r.a, r.d, x * m + y)));
      }
      std::sort(img.begin(), img.end());
      if (img < f) smallest = false;
      int gpos = 0;
      while (gpos < n_groups && ++pick[gpos] == (int)perms.size()) pick[gpos++] = 0;
      if (gpos == n_groups) break;
    }
    if (smallest) out.push_back(f);
  }
  return out;
}

// Family-level pruning (Sec. 4.1): inside one shape bucket, exact duplicates
// (the same multiset of (group pair, footprint, rate), e.g. two PIX copies
// swapped) collapse to the first family in canonical order, and a family is
// removed when another one of the bucket dominates it: their instances pair
// up inside every group pair with identical footprints and no lower rate,
// with at least one strictly higher rate.
std::vector<Fam> drop_duplicate_and_dominated(std::vector<Fam> fams, const std::vector<Inst>& table) {
  std::sort(fams.begin(), fams.end());
  typedef std::tuple<int, int, bool, std::vector<int>> PairFoot;
  auto rates_by_foot = [&](const Fam& f) {
    std::map<PairFoot, std::vector<i64>> m;
    for (int id : f) {
      const Inst& r = table[id];
      m[PairFoot(r.a, r.d, r.remote, r.L)].push_back(r.bw);
    }
    for (auto& kv : m) std::sort(kv.second.rbegin(), kv.second.rend());
    return m;
  };
  std::vector<Fam> uniq;
  std::vector<std::map<PairFoot, std::vector<i64>>> prof;
  std::set<std::map<PairFoot, std::vector<i64>>> seen;
  for (const Fam& f : fams) {
    auto m = rates_by_foot(f);
    if (seen.insert(m).second) {
      uniq.push_back(f);
      prof.push_back(m);
    }
  }
  // y dominates x: same (group pair, footprint) classes with the same sizes,
  // rates sorted descending pairwise no lower, one strictly higher
  auto dominates = [&](size_t y, size_t x) {
    if (prof[y].size() != prof[x].size()) return false;
    bool higher = false;
    for (const auto& kv : prof[x]) {
      auto it = prof[y].find(kv.first);
      if (it == prof[y].end() || it->second.size() != kv.second.size()) return false;
      for (size_t u = 0; u < kv.second.size(); ++u) {
        if (it->second[u] < kv.second[u]) return false;
        higher |= it->second[u] > kv.second[u];
      }
    }
    return higher;
  };
  std::vector<Fam> out;
  for (size_t x = 0; x < uniq.size(); ++x) {
    bool dom = false;
    for (size_t y = 0; y < uniq.size() && !dom; ++y) dom = y != x && dominates(y, x);
    if (!dom) out.push_back(uniq[x]);
  }
  return out;
}

// The catalog of one instance set: drop dominated paths, find every family,
// file each under its shape (lane counts per group pair, remote lanes
// counted apart), then prune each bucket and keep one family per NIC
// renaming.
std::map<ShapeKey, std::vector<Fam>> catalog_of(const std::vector<Inst>& table,
                                                const std::vector<Inst>& candidates, int n_groups, int g,
                                                int n_res, int nics) {
  std::vector<Inst> R = drop_dominated_paths(candidates);
  std::sort(R.begin(), R.end(), [](const Inst& x, const Inst& y) { return x.id < y.id; });
  std::map<ShapeKey, std::vector<Fam>> buckets;
  for (const auto& sel : all_families(R, n_groups, g, n_res)) {
    ShapeKey M(2 * n_groups * n_groups, 0);
    Fam f;
    for (int i : sel) {
      const Inst& r = R[i];
      M[(r.remote ? n_groups * n_groups : 0) + r.a * n_groups + r.d]++;
      f.push_back(r.id);
    }
    std::sort(f.begin(), f.end());
    buckets[M].push_back(f);
  }
  for (auto& kv : buckets)
    kv.second = keep_nic_canonical(drop_duplicate_and_dominated(kv.second, table), table, n_groups, nics);
  return buckets;
}

// ---------------------------------------------------------------------------
// Catalog at cluster level: what Alg. 2 consumes.
// ---------------------------------------------------------------------------
struct CInst {
  int a, d;      // source / destination group
  int cls;
  i64 bw;
  int id;        // instance id recorded in the schedule
};
struct CFamily {
  int shape;
  int k;                       // node shift (node-circulant catalogs)
  std::vector<int> local;      // node-local instance ids (node-circulant catalogs)
  std::vector<CInst> inst;     // N instances in family order
};
struct CShape {
  int k;
  std::vector<int> Lm, Rm;                        // Q x Q block counts (circulant)
  std::vector<std::tuple<int, int, int>> M;       // nonzero (a, d, M_ad)
  std::vector<int> dense;                         // G x G (full catalogs only)
  int fam_begin, fam_end;
};

struct Catalog {
  Topo topo;
  bool circulant;
  std::vector<Inst> table;       // instance table (node-local or cluster)
  std::vector<CShape> shapes;
  std::vector<CFamily> fams;
  i64 bw_max;
};

// The nearest path of an ordered group pair (Sec. 6.3 peer/path ablation,
// "fixed nearest path"): PIX inside a switch, PXB between two switches of one
// socket, SYS between sockets of one node when enabled, the NICs otherwise.
// A family keeps only lanes on their pair's nearest path; under the topology
// model the only other choice is a NIC lane between two switches of one node
// that a PXB (or SYS) path also joins.  Group ids are node-major, so
// a / Q is the node and (a % Q) / switches the socket.
bool nearest_only(const std::vector<Inst>& table, const Fam& f, const Topo& t, bool remote_set) {
  const int Q = t.Q();
  for (int id : f) {
    const Inst& r = table[id];
    if (r.cls != NIC || remote_set || r.a == r.d || r.a / Q != r.d / Q) continue;
    const bool same_socket = (r.a % Q) / t.switches == (r.d % Q) / t.switches;
    if (same_socket || t.sys) return false;
  }
  return true;
}

void keep_nearest(std::map<ShapeKey, std::vector<Fam>>& b, const std::vector<Inst>& table, const Topo& t,
                  bool remote_set) {
  for (auto it = b.begin(); it != b.end();) {
    std::vector<Fam> keep;
    for (const Fam& f : it->second)
      if (nearest_only(table, f, t, remote_set)) keep.push_back(f);
    if (keep.empty()) it = b.erase(it);
    else { it->second = keep; ++it; }
  }
}

// Node-circulant catalog: a family is (k, B_loc): the same node-local pattern
// in every node, NIC lanes of node n landing on node (n + k) mod n_nodes; k = 0
// holds every family whose NIC lanes (if any) stay inside the node.  With one
// node this is exactly Alg. 1's catalog.
void build_circulant(Catalog& C, bool nearest) {
  const Topo& t = C.topo;
  const int Q = t.Q(), g = t.g, nn = t.n_nodes;
  C.table = local_table(t);
  const int n_res = 2 * Q + 2 * Q * t.nics + t.sockets * t.sockets;
  // k = 0 set: PIX, PXB, NIC between slots of the same node (loopback).
  std::vector<Inst> set0;
  for (Inst r : C.table) { r.remote = false; set0.push_back(r); }
  auto b0 = catalog_of(C.table, set0, Q, g, n_res, t.nics);
  if (nearest) keep_nearest(b0, C.table, t, false);
  // k != 0 set: PIX, PXB, and NIC lanes to the same slot pattern on another node.
  std::map<ShapeKey, std::vector<Fam>> b1;
  if (nn > 1) {
    std::vector<Inst> set1;
    for (Inst r : C.table) { r.remote = (r.cls == NIC); set1.push_back(r); }
    std::vector<Inst> table1 = set1;
    auto all1 = catalog_of(table1, set1, Q, g, n_res, t.nics);
    for (auto& kv : all1) {
      std::vector<Fam> keep;
      for (const Fam& f : kv.second) {
        bool has_nic = false;
        for (int id : f) has_nic |= C.table[id].cls == NIC;
        if (has_nic) keep.push_back(f);       // NIC-free families live under k = 0
      }
      if (!keep.empty()) b1[kv.first] = keep;
    }
  }
  // Canonical order: shapes by (k, diagonal-block counts, shift-block counts),
  // families by their sorted instance ids.  std::map keys are the row-major
  // (diagonal block, shift block) counts, so iteration order is canonical.
  auto emit = [&](int k, const std::map<ShapeKey, std::vector<Fam>>& b) {
    for (const auto& kv : b) {
      CShape s;
      s.k = k;
      s.Lm.assign(kv.first.begin(), kv.first.begin() + Q * Q);
      s.Rm.assign(kv.first.begin() + Q * Q, kv.first.end());
      std::map<std::pair<int, int>, int> m;
      for (int n = 0; n < nn; ++n)
        for (int q = 0; q < Q; ++q)
          for (int q2 = 0; q2 < Q; ++q2) {
            if (s.Lm[q * Q + q2]) m[{n * Q + q, n * Q + q2}] += s.Lm[q * Q + q2];
            if (s.Rm[q * Q + q2]) m[{n * Q + q, ((n + k) % nn) * Q + q2}] += s.Rm[q * Q + q2];
          }
      for (auto& e : m) s.M.emplace_back(e.first.first, e.first.second, e.second);
      s.fam_begin = (int)C.fams.size();
      std::vector<Fam> fs = kv.second;
      std::sort(fs.begin(), fs.end());
      for (const Fam& f : fs) {
        CFamily F;
        F.shape = (int)C.shapes.size();
        F.k = k;
        F.local = f;
        for (int n = 0; n < nn; ++n)
          for (int id : f) {
            const Inst& r = C.table[id];
            int dn = (r.cls == NIC && k != 0) ? (n + k) % nn : n;
            F.inst.push_back({n * Q + r.a, dn * Q + r.d, r.cls, r.bw, id});
          }
        C.fams.push_back(F);
      }
      s.fam_end = (int)C.fams.size();
      C.shapes.push_back(s);
    }
  };
  emit(0, b0);
  for (int k = 1; k < nn; ++k) emit(k, b1);
}

// Full Alg. 1 over the cluster-level instance set (small topologies only).
void build_full(Catalog& C, bool nearest) {
  const Topo& t = C.topo;
  const int G = t.G();
  C.table = cluster_table(t);
  auto b = catalog_of(C.table, C.table, G, t.g, 2 * G + 2 * G * t.nics + t.n_nodes * t.sockets * t.sockets, t.nics);
  if (nearest) keep_nearest(b, C.table, t, false);
  for (const auto& kv : b) {
    CShape s;
    s.k = -1;
    s.dense.assign(kv.first.begin(), kv.first.begin() + G * G);
    for (int a = 0; a < G; ++a)
      for (int d = 0; d < G; ++d)
        if (s.dense[a * G + d]) s.M.emplace_back(a, d, s.dense[a * G + d]);
    s.fam_begin = (int)C.fams.size();
    for (const Fam& f : kv.second) {
      CFamily F;
      F.shape = (int)C.shapes.size();
      F.k = -1;
      F.local = f;
      for (int id : f) {
        const Inst& r = C.table[id];
        F.inst.push_back({r.a, r.d, r.cls, r.bw, id});
      }
      C.fams.push_back(F);
    }
    s.fam_end = (int)C.fams.size();
    C.shapes.push_back(s);
  }
}

// ---------------------------------------------------------------------------
// Counter-based randomness for the random AA starts: SplitMix64 (Steele, Lea
// and Flood, OOPSLA 2014).  The key absorbs (seed, iteration, family, start,
// group, side) one field at a time; the stream then steps the SplitMix64 state.
// ---------------------------------------------------------------------------
const uint64_t GOLDEN = 0x9E3779B97F4A7C15ULL;
uint64_t sm_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
  return z ^ (z >> 31);
}
struct SplitMix {
  uint64_t state;
  uint64_t next() { state += GOLDEN; return sm_mix(state); }
};
SplitMix keyed_stream(uint64_t seed, uint64_t iter, uint64_t fam, uint64_t start,
                      uint64_t group, uint64_t side) {
  uint64_t key = seed;
  const uint64_t fields[5] = {iter, fam, start, group, side};
  for (uint64_t v : fields) key = sm_mix(key + GOLDEN) ^ v;
  return SplitMix{key};
}

// ---------------------------------------------------------------------------
// Online channel-guided demand decomposition (Sec. 4.2, Alg. 2).
// ---------------------------------------------------------------------------
struct Params {
  i64 k_target, lambda_ns, unit;
  int n_start, i_aa;
  uint64_t seed;
};

struct Planner {
  const Catalog& C;
  const Params& P;
  int N, G, g;
  std::vector<i64> Drem;           // D^rem, row-major N x N bytes
  i64 tau;
  i64 K;                           // activations emitted so far
  // optional trace of F after every AA half-step: (iter, family, start, half, F)
  i64* trace;
  i64 trace_cap, trace_n;
  // optional log of every evaluated candidate: (iter, family, S, x, b, then
  // per instance in family order: source, destination, volume)
  i64* cand_log;
  i64 cand_cap, cand_n;

  Planner(const Catalog& C_, const Params& P_) : C(C_), P(P_) {
    N = C.topo.N();
    G = C.topo.G();
    g = C.topo.g;
    trace = nullptr;
    trace_cap = trace_n = 0;
    cand_log = nullptr;
    cand_cap = cand_n = 0;
    K = 0;
    tau = 1;
  }

  // Capacity of a path within one quantum, rounded down to whole units
  // (at least one unit): the integer form of tau * bw(p) in Eq. (9).
  i64 cap(i64 bw) const {
    i64 c = (tau * bw) / P.unit * P.unit;
    return c < P.unit ? P.unit : c;
  }

  // Binding credit, Eq. (7), scaled by tau: h' = min(D^rem_ij, tau*bw(r)).
  // Self pairs lie outside Gamma_ad and are never bound.
  i64 credit(const CInst& r, int i, int j) const {
    i64 dv = Drem[(size_t)i * N + j];
    i64 c = cap(r.bw);
    return dv < c ? dv : c;
  }

  struct Binding { std::vector<int> src, dst; };

  // Out-instances / in-instances of every group, in family order.
  void group_lists(const CFamily& F, std::vector<std::vector<int>>& outs,
                   std::vector<std::vector<int>>& ins) const {
    outs.assign(G, {});
    ins.assign(G, {});
    for (int t = 0; t < (int)F.inst.size(); ++t) {
      outs[F.inst[t].a].push_back(t);
      ins[F.inst[t].d].push_back(t);
    }
  }

  // Binding score, Eq. (8): sum of the bound credits.
  i64 score(const CFamily& F, const Binding& b) const {
    i64 s = 0;
    for (int t = 0; t < (int)F.inst.size(); ++t) s += credit(F.inst[t], b.src[t], b.dst[t]);
    return s;
  }

  // Make the binding self-transfer free (Gamma_ad excludes i == j): for every
  // group, walk its intra-group instances in family order; a self-bound one
  // trades destinations with the first other in-instance of the group that is
  // not protected, or, failing that, sources with the first other unprotected
  // out-instance.  A trade never creates a new self-binding.
  void repair(const CFamily& F, Binding& b, int protect,
              const std::vector<std::vector<int>>& outs,
              const std::vector<std::vector<int>>& ins) const {
    for (int a = 0; a < G; ++a) {
      for (int r : outs[a]) {
        if (F.inst[r].d != a || b.src[r] != b.dst[r]) continue;
        int partner = -1;
        for (int r2 : ins[a])
          if (r2 != r && r2 != protect) { partner = r2; break; }
        if (partner >= 0) {
          std::swap(b.dst[r], b.dst[partner]);
          continue;
        }
        for (int r3 : outs[a])
          if (r3 != r && r3 != protect) { partner = r3; break; }
        if (partner >= 0) std::swap(b.src[r], b.src[partner]);
      }
    }
  }

  // Start 0: the canonical binding (the g out-instances of group a take
  // sources a*g+0.., the g in-instances of group d take destinations d*g+0..,
  // both in family order) with the single highest-credit triple (t, i, j)
  // forced in; ties go to the smallest (t, i, j).
  Binding start_forced(const CFamily& F, const std::vector<std::vector<int>>& outs,
                       const std::vector<std::vector<int>>& ins) const {
    const int n = (int)F.inst.size();
    Binding b;
    b.src.assign(n, -1);
    b.dst.assign(n, -1);
    for (int a = 0; a < G; ++a)
      for (int m = 0; m < (int)outs[a].size(); ++m) b.src[outs[a][m]] = a * g + m;
    for (int d = 0; d < G; ++d)
      for (int m = 0; m < (int)ins[d].size(); ++m) b.dst[ins[d][m]] = d * g + m;
    i64 best = 0;
    int bt = -1, bi = -1, bj = -1;
    for (int t = 0; t < n; ++t)
      for (int il = 0; il < g; ++il)
        for (int jl = 0; jl < g; ++jl) {
          int i = F.inst[t].a * g + il, j = F.inst[t].d * g + jl;
          if (i == j) continue;
          i64 h = credit(F.inst[t], i, j);
          if (h > best) { best = h; bt = t; bi = i; bj = j; }
        }
    int protect = -1;
    if (bt >= 0) {
      for (int t2 : outs[F.inst[bt].a])
        if (b.src[t2] == bi) { std::swap(b.src[t2], b.src[bt]); break; }
      for (int t3 : ins[F.inst[bt].d])
        if (b.dst[t3] == bj) { std::swap(b.dst[t3], b.dst[bt]); break; }
      protect = bt;
    }
    repair(F, b, protect, outs, ins);
    return b;
  }

  // Starts 1..N_start-1: an independent Fisher-Yates shuffle of every group's
  // sources and of every group's destinations, then the self-binding repair.
  Binding start_random(const CFamily& F, int fam_index, int s,
                       const std::vector<std::vector<int>>& outs,
                       const std::vector<std::vector<int>>& ins) const {
    const int n = (int)F.inst.size();
    Binding b;
    b.src.assign(n, -1);
    b.dst.assign(n, -1);
    for (int side = 0; side < 2; ++side)
      for (int x = 0; x < G; ++x) {
        SplitMix rng = keyed_stream(P.seed, (uint64_t)K, (uint64_t)fam_index, (uint64_t)s,
                                    (uint64_t)x, (uint64_t)side);
        std::vector<int> perm(g);
        for (int m = 0; m < g; ++m) perm[m] = m;
        for (int m = g - 1; m >= 1; --m) {
          int j = (int)(rng.next() % (uint64_t)(m + 1));
          std::swap(perm[m], perm[j]);
        }
        const std::vector<int>& lst = side == 0 ? outs[x] : ins[x];
        for (int m = 0; m < (int)lst.size(); ++m) {
          if (side == 0) b.src[lst[m]] = x * g + perm[m];
          else b.dst[lst[m]] = x * g + perm[m];
        }
      }
    repair(F, b, -1, outs, ins);
    return b;
  }

  // One half of an AA sweep for one group: with the other side fixed, try
  // every assignment of the group's g ranks to its g instances (lexicographic
  // order of the rank tuple), skip those that bind a rank to itself, and take
  // the first best one if it strictly beats the current assignment.
  bool improve_group(const CFamily& F, Binding& b, const std::vector<int>& lst, int x,
                     bool source_side) const {
    std::vector<int> perm(g);
    for (int m = 0; m < g; ++m) perm[m] = m;
    i64 cur = 0;
    for (int t : lst) cur += credit(F.inst[t], b.src[t], b.dst[t]);
    i64 best = -1;
    std::vector<int> best_perm;
    do {
      bool ok = true;
      i64 v = 0;
      for (int m = 0; m < g && ok; ++m) {
        int t = lst[m];
        int i = source_side ? x * g + perm[m] : b.src[t];
        int j = source_side ? b.dst[t] : x * g + perm[m];
        if (i == j) { ok = false; break; }
        v += credit(F.inst[t], i, j);
      }
      if (ok && v > best) { best = v; best_perm = perm; }
    } while (std::next_permutation(perm.begin(), perm.end()));
    if (best > cur) {
      for (int m = 0; m < g; ++m) {
        if (source_side) b.src[lst[m]] = x * g + best_perm[m];
        else b.dst[lst[m]] = x * g + best_perm[m];
      }
      return true;
    }
    return false;
  }

  void log(int f, int s, int half, i64 F) {
    if (!trace || trace_n >= trace_cap) return;
    i64* e = trace + 5 * trace_n;
    e[0] = K; e[1] = f; e[2] = s; e[3] = half; e[4] = F;
    ++trace_n;
  }

  // Alternating Algorithm (Sec. 4.2 Step 2): source half, then destination
  // half; each solves one g x g assignment per group without decreasing F_B.
  // Stop after I_AA sweeps or after a sweep that changes nothing.
  void alternating(const CFamily& F, int f, int s, Binding& b,
                   const std::vector<std::vector<int>>& outs,
                   const std::vector<std::vector<int>>& ins) {
    log(f, s, 0, score(F, b));
    for (int sweep = 0; sweep < P.i_aa; ++sweep) {
      bool changed = false;
      for (int a = 0; a < G; ++a) changed |= improve_group(F, b, outs[a], a, true);
      log(f, s, 2 * sweep + 1, score(F, b));
      for (int d = 0; d < G; ++d) changed |= improve_group(F, b, ins[d], d, false);
      log(f, s, 2 * sweep + 2, score(F, b));
      if (!changed) break;
    }
  }

  // MultiStartAA: run AA from N_start feasible bindings and keep the highest
  // F_B (ties to the earliest start).
  Binding multistart_aa(const CFamily& F, int f) {
    std::vector<std::vector<int>> outs, ins;
    group_lists(F, outs, ins);
    Binding best;
    i64 bestF = -1;
    for (int s = 0; s < P.n_start; ++s) {
      Binding b = s == 0 ? start_forced(F, outs, ins) : start_random(F, f, s, outs, ins);
      alternating(F, f, s, b, outs, ins);
      i64 Fb = score(F, b);
      if (Fb > bestF) { bestF = Fb; best = b; }
    }
    return best;
  }

  // Evaluate (Sec. 4.2 Step 3): lane volumes by Eq. (9) and the utility of
  // Eq. (10) kept as (S, x, b) with U = S / (lambda + x / b).
  struct Eval { std::vector<i64> x; i64 S, xm, bm; };
  Eval evaluate(const CFamily& F, const Binding& b) const {
    Eval e;
    const int n = (int)F.inst.size();
    e.x.assign(n, 0);
    e.S = 0;
    e.xm = 0;
    e.bm = 1;
    std::vector<int> by_rank(N, -1);
    for (int t = 0; t < n; ++t) {
      i64 c = cap(F.inst[t].bw);
      i64 dv = Drem[(size_t)b.src[t] * N + b.dst[t]];
      e.x[t] = c < dv ? c : dv;
      e.S += e.x[t];
      by_rank[b.src[t]] = t;
    }
    for (int i = 0; i < N; ++i) {        // slowest lane; ties to the lowest rank
      int t = by_rank[i];
      if ((u128)e.x[t] * (u128)e.bm > (u128)e.xm * (u128)F.inst[t].bw) {
        e.xm = e.x[t];
        e.bm = F.inst[t].bw;
      }
    }
    return e;
  }

  // U_1 > U_2 exactly.  U = 0 when S = 0.
  bool better(const Eval& e1, const Eval& e2) const {
    if (e1.S == 0) return false;
    if (e2.S == 0) return true;
    u128 lam = (u128)P.lambda_ns;
    u128 lhs = (u128)e1.S * (u128)e1.bm * (lam * (u128)e2.bm + (u128)e2.xm);
    u128 rhs = (u128)e2.S * (u128)e2.bm * (lam * (u128)e1.bm + (u128)e1.xm);
    return lhs > rhs;
  }

  // Take D as the residual: every entry non-negative, a whole number of
  // units and zero on the diagonal (Sec. 3: self traffic stays local).
  bool load(const i64* D) {
    Drem.assign(D, D + (size_t)N * N);
    for (int i = 0; i < N; ++i)
      for (int j = 0; j < N; ++j) {
        const i64 v = Drem[(size_t)i * N + j];
        if (v < 0 || v % P.unit != 0 || (i == j && v != 0)) return false;
      }
    return true;
  }

  // Global time quantum (Sec. 5 "Global execution granularity"): the most
  // loaded rank (largest row or column sum) drains in about K_target quanta
  // at the fastest path rate.
  void set_quantum() {
    i64 heaviest = 0;
    for (int i = 0; i < N; ++i) {
      i64 out = 0, in = 0;
      for (int j = 0; j < N; ++j) {
        out += Drem[(size_t)i * N + j];
        in += Drem[(size_t)j * N + i];
      }
      heaviest = std::max(heaviest, std::max(out, in));
    }
    const i64 per_quantum = C.bw_max * P.k_target;
    tau = std::max<i64>(1, (heaviest + per_quantum - 1) / per_quantum);
  }

  i64 unserved() const {
    i64 s = 0;
    for (i64 v : Drem) s += v;
    return s;
  }

  // Step 1 (Eq. (5), Eq. (6)): the residual summed per ordered group pair,
  // then the shape whose lane counts weigh it most; the first such shape in
  // canonical order, or -1 when every score is zero.
  int pressure_argmax() const {
    std::vector<i64> Dhat((size_t)G * G, 0);
    for (int i = 0; i < N; ++i)
      for (int j = 0; j < N; ++j) Dhat[(size_t)(i / g) * G + j / g] += Drem[(size_t)i * N + j];
    int arg = -1;
    i64 top = 0;
    for (int m = 0; m < (int)C.shapes.size(); ++m) {
      i64 sc = 0;
      for (const auto& e : C.shapes[m].M)
        sc += Dhat[(size_t)std::get<0>(e) * G + std::get<1>(e)] * std::get<2>(e);
      if (sc > top) {
        top = sc;
        arg = m;
      }
    }
    return arg;
  }

  // Steps 2 and 3 for one family of the chosen shape: its best binding over
  // the starts, then the lane volumes and utility of that channel.
  struct Candidate {
    int f;
    Binding b;
    Eval e;
  };
  Candidate candidate_for(int f) {
    Candidate c;
    c.f = f;
    c.b = multistart_aa(C.fams[f], f);
    c.e = evaluate(C.fams[f], c.b);
    if (cand_log && cand_n < cand_cap) {
      const size_t w = 5 + 3 * (size_t)N;
      i64* r = cand_log + w * (size_t)cand_n++;
      r[0] = K; r[1] = f; r[2] = c.e.S; r[3] = c.e.xm; r[4] = c.e.bm;
      for (int t = 0; t < (int)C.fams[f].inst.size(); ++t) {
        r[5 + 3 * t] = c.b.src[t];
        r[6 + 3 * t] = c.b.dst[t];
        r[7 + 3 * t] = c.e.x[t];
      }
    }
    return c;
  }

  // The activation joins the schedule and its volumes leave the residual.
  void commit(const Candidate& c, int32_t* fam, int32_t* dst, int32_t* inst, i64* bytes) {
    const CFamily& F = C.fams[c.f];
    fam[K] = c.f;
    for (int t = 0; t < (int)F.inst.size(); ++t) {
      const int i = c.b.src[t], j = c.b.dst[t];
      const size_t o = (size_t)K * N + i;
      dst[o] = j;
      inst[o] = F.inst[t].id;
      bytes[o] = c.e.x[t];
      Drem[(size_t)i * N + j] -= c.e.x[t];
    }
    ++K;
  }

  // The activation a shape yields: every family's candidate, the one with
  // the highest utility kept (the first in canonical order on ties).
  Candidate best_candidate(int m) {
    Candidate win;
    win.f = -1;
    for (int f = C.shapes[m].fam_begin; f < C.shapes[m].fam_end; ++f) {
      Candidate c = candidate_for(f);
      if (win.f < 0 || better(c.e, win.e)) win = c;
    }
    return win;
  }

  // The decomposition (Sec. 4.2): until nothing is left, pick the shape,
  // take the best activation it yields and commit it.  K_max bounds the
  // schedule.
  int run(const i64* D, int32_t* Kout, int32_t* fam, int32_t* dst, int32_t* inst,
          i64* bytes, int k_max, i64* tau_out) {
    *Kout = 0;
    K = 0;
    if (!load(D)) return INVALID_DEMAND;
    set_quantum();
    if (tau_out) *tau_out = tau;
    for (;;) {
      if (unserved() == 0) return OK;
      if (K >= k_max) return CAPACITY;
      const int m = pressure_argmax();
      if (m < 0) return NO_PROGRESS;
      const Candidate win = best_candidate(m);
      if (win.f < 0 || win.e.S == 0) return NO_PROGRESS;
      commit(win, fam, dst, inst, bytes);
      *Kout = (int32_t)K;
    }
  }
};

}  // namespace

// ===========================================================================
// C interface for the Python side (ctypes).
// ===========================================================================
extern "C" {

struct orc_catalog;   // opaque: a Catalog

struct orc_topology {
  int32_t n_nodes, sockets_per_node, switches_per_socket, gpus_per_switch, nics_per_switch;
  int32_t flags;   // bit 0: peer to peer between sockets (SYS paths)
  int64_t pcie_bytes_per_ns, nic_bytes_per_ns;
};

struct orc_params {
  int64_t k_target, lambda_ns, unit_bytes;
  int32_t n_start, i_aa;
  uint64_t seed;
};

// mode bit 0 clear: node-circulant catalog (equal to full Alg. 1 for one node)
// mode bit 0 set:   full Alg. 1 over the cluster-level instance set (small topologies)
// mode bit 1 set:   only families whose lanes all take their pair's nearest path
int orc_catalog_build(const orc_topology* tp, int mode, orc_catalog** out) {
  if (!tp || !out) return INVALID_ARGUMENT;
  Topo t{tp->n_nodes, tp->sockets_per_node, tp->switches_per_socket, tp->gpus_per_switch,
         tp->nics_per_switch, tp->pcie_bytes_per_ns, tp->nic_bytes_per_ns, (tp->flags & 1) != 0};
  // every ordered pair needs a path: 1 to 4 NICs per switch, at least two GPUs per switch
  if (t.n_nodes < 1 || t.sockets < 1 || t.switches < 1 || t.g < 2 || t.nics < 1 || t.nics > 4 ||
      t.pcie < 1 || t.nic < 1 || (tp->flags & ~1) != 0)
    return INVALID_ARGUMENT;
  Catalog* C = new Catalog();
  C->topo = t;
  C->circulant = (mode & 1) == 0;
  if (mode & ~3) { delete C; return INVALID_ARGUMENT; }
  if (C->circulant) build_circulant(*C, (mode & 2) != 0);
  else build_full(*C, (mode & 2) != 0);
  C->bw_max = 0;
  for (const auto& r : C->table) C->bw_max = std::max(C->bw_max, r.bw);
  *out = reinterpret_cast<orc_catalog*>(C);
  return OK;
}

void orc_catalog_free(orc_catalog* c) { delete reinterpret_cast<Catalog*>(c); }

// info[0..7] = N, G, g, Q, n_nodes, n_shapes, n_families, n_table_instances
int orc_catalog_info(const orc_catalog* c, int64_t* info) {
  const Catalog* C = reinterpret_cast<const Catalog*>(c);
  info[0] = C->topo.N();
  info[1] = C->topo.G();
  info[2] = C->topo.g;
  info[3] = C->topo.Q();
  info[4] = C->topo.n_nodes;
  info[5] = (int64_t)C->shapes.size();
  info[6] = (int64_t)C->fams.size();
  info[7] = (int64_t)C->table.size();
  return OK;
}

// Instance table: class, src, dst, copy, rate, and up to 2 resource ids (-1 pad).
int orc_catalog_table(const orc_catalog* c, int32_t* cls, int32_t* src, int32_t* dst,
                      int32_t* copy, int64_t* bw, int32_t* res2) {
  const Catalog* C = reinterpret_cast<const Catalog*>(c);
  for (size_t i = 0; i < C->table.size(); ++i) {
    const Inst& r = C->table[i];
    cls[i] = r.cls; src[i] = r.a; dst[i] = r.d; copy[i] = r.copy; bw[i] = r.bw;
    res2[2 * i] = r.L.size() > 0 ? r.L[0] : -1;
    res2[2 * i + 1] = r.L.size() > 1 ? r.L[1] : -1;
  }
  return OK;
}

// Shapes: k, bucket range; circulant: Q x Q diagonal/shift blocks;
// full: dense G x G written to Lm (Rm untouched).
int orc_catalog_shapes(const orc_catalog* c, int32_t* k, int32_t* fam_begin, int32_t* fam_end,
                       int32_t* Lm, int32_t* Rm) {
  const Catalog* C = reinterpret_cast<const Catalog*>(c);
  const int Q = C->topo.Q(), G = C->topo.G();
  for (size_t m = 0; m < C->shapes.size(); ++m) {
    const CShape& s = C->shapes[m];
    k[m] = s.k;
    fam_begin[m] = s.fam_begin;
    fam_end[m] = s.fam_end;
    if (C->circulant) {
      for (int x = 0; x < Q * Q; ++x) { Lm[m * Q * Q + x] = s.Lm[x]; Rm[m * Q * Q + x] = s.Rm[x]; }
    } else {
      for (int x = 0; x < G * G; ++x) Lm[m * G * G + x] = s.dense[x];
    }
  }
  return OK;
}

// Families: shape, k, and the instance ids (local ids for circulant
// catalogs: Q*g per family; cluster ids for full catalogs: N per family).
int orc_catalog_families(const orc_catalog* c, int32_t* shape, int32_t* k, int32_t* ids) {
  const Catalog* C = reinterpret_cast<const Catalog*>(c);
  size_t w = C->fams.empty() ? 0 : C->fams[0].local.size();
  for (size_t f = 0; f < C->fams.size(); ++f) {
    shape[f] = C->fams[f].shape;
    k[f] = C->fams[f].k;
    for (size_t x = 0; x < w; ++x) ids[f * w + x] = C->fams[f].local[x];
  }
  return OK;
}

// Cluster view of one family: per instance t (family order): class, source
// group, destination group, recorded id.
int orc_catalog_cluster_family(const orc_catalog* c, int32_t f, int32_t* cls, int32_t* a,
                               int32_t* d, int32_t* id) {
  const Catalog* C = reinterpret_cast<const Catalog*>(c);
  if (f < 0 || f >= (int32_t)C->fams.size()) return INVALID_ARGUMENT;
  const CFamily& F = C->fams[f];
  for (size_t t = 0; t < F.inst.size(); ++t) {
    cls[t] = F.inst[t].cls; a[t] = F.inst[t].a; d[t] = F.inst[t].d; id[t] = F.inst[t].id;
  }
  return OK;
}

// Demand row of one source rank (Sec. 3 model setup; Sec. 5 sparse EP):
// counts[e] = #{(t, e)}; D_self,j = unit * sum of counts of the experts that
// rank j hosts (experts are contiguous per rank), D_self,self = 0.  Also the
// stable (expert, token) order of the assignments (token and routing slot of
// each) and each destination's first row in it.
int orc_demand(const int32_t* routing, int64_t T, int32_t k, int32_t E, int32_t N,
               int32_t self, int64_t unit, int64_t* row, int32_t* counts, int32_t* sorted_tok,
               uint8_t* sorted_slot, int64_t* dest_off) {
  if (N < 1 || E < N || E % N != 0 || self < 0 || self >= N || unit < 1) return INVALID_ARGUMENT;
  const int eloc = E / N;
  for (int e = 0; e < E; ++e) counts[e] = 0;
  for (int64_t x = 0; x < T * k; ++x) {
    int e = routing[x];
    if (e < 0 || e >= E) return INVALID_ARGUMENT;
    counts[e]++;
  }
  for (int j = 0; j < N; ++j) {
    int64_t c = 0;
    for (int e = j * eloc; e < (j + 1) * eloc; ++e) c += counts[e];
    row[j] = j == self ? 0 : c * unit;
  }
  // stable order by expert: walk experts ascending, tokens ascending
  std::vector<int64_t> start(E + 1, 0);
  for (int e = 0; e < E; ++e) start[e + 1] = start[e] + counts[e];
  std::vector<int64_t> fill(start.begin(), start.end() - 1);
  // each entry is one (token, slot) assignment: its token, and which of the
  // token's k routing slots it is
  for (int64_t x = 0; x < T * k; ++x) {
    int e = routing[x];
    if (sorted_slot) sorted_slot[fill[e]] = (uint8_t)(x % k);
    sorted_tok[fill[e]++] = (int32_t)(x / k);
  }
  for (int j = 0; j <= N; ++j) dest_off[j] = start[(size_t)j * eloc];
  return OK;
}

// Sparse expert-parallel control words (Sec. 5, efficient sparse data
// movement for expert parallelism), one source rank's row.  Destination j
// hosts L = E/N local experts (experts j*L .. j*L+L-1).  For an active pair
// the 32-bit word has bit l set when the source sends at least one row to
// local expert l, and the bits above the L bitmap bits hold the exact row
// count of the designated expert.  Reading: the designated expert is the
// highest active one, because the pair's stream runs expert-ascending and
// the word travels right after that expert's payload.  Pairs with no rows
// and the self pair get no word (0).
int orc_control_words(const int32_t* counts, int32_t E, int32_t N, int32_t self, uint32_t* words) {
  if (N < 1 || E < N || E % N != 0 || self < 0 || self >= N) return INVALID_ARGUMENT;
  const int L = E / N;
  if (L > 31) return UNSUPPORTED;
  for (int j = 0; j < N; ++j) {
    words[j] = 0;
    if (j == self) continue;
    uint32_t bitmap = 0;
    int designated = -1;
    for (int l = 0; l < L; ++l) {
      const int32_t c = counts[j * L + l];
      if (c < 0) return INVALID_ARGUMENT;
      if (c > 0) {
        bitmap |= 1u << l;
        designated = l;
      }
    }
    if (designated < 0) continue;
    const uint64_t c = (uint64_t)counts[j * L + designated];
    if (c >= (1ull << (32 - L))) return CAPACITY;   // the count field has 32 - L bits
    words[j] = bitmap | (uint32_t)(c << L);
  }
  return OK;
}

// The receiving side of the same words: rank r rebuilds the rows it gets from
// every source for each of its L local experts.  An expert whose bitmap bit
// is clear gets nothing (it is skipped); the designated expert's count comes
// from the word; the other active experts' counts come from the per-expert
// completion signals (`signal` [N][L], read only for those entries).
int orc_receive_counts(const uint32_t* words, const int32_t* signal, int32_t N, int32_t L,
                       int32_t* counts) {
  if (N < 1 || L < 1 || L > 31) return INVALID_ARGUMENT;
  for (int i = 0; i < N; ++i) {
    const uint32_t w = words[i];
    const uint32_t bitmap = w & ((1u << L) - 1);
    int designated = -1;
    for (int l = 0; l < L; ++l)
      if (bitmap >> l & 1) designated = l;
    for (int l = 0; l < L; ++l) {
      int32_t c = 0;
      if (l == designated) c = (int32_t)(w >> L);
      else if (bitmap >> l & 1) c = signal[i * L + l];
      counts[i * L + l] = c;
    }
  }
  return OK;
}

// Fixed cyclic peer rotation, the baseline of the peer/path ablation
// (Sec. 6.3, Table 3).  Stage s = 1..N-1: rank i sends all of D_i,(i+s mod N)
// at once; empty stages are skipped.  Each lane uses its pair's nearest path
// (nearest = 1) or, per stage, the path vector that ends the stage first
// (nearest = 0), every vector tried.  Lanes sharing a directed resource
// split its capacity equally: a lane's rate is the least of its path rate
// and capacity / sharers over its resources (UP and DN links and the socket
// link carry the PCIe rate, TX and RX the NIC rate).  Stage time = lambda + max bytes / rate.
// The result is the exact rational total in ns.
int orc_rotation_time(const orc_topology* tp, const int64_t* D, int32_t nearest, int64_t lambda,
                      int64_t* num, int64_t* den) {
  Topo t{tp->n_nodes, tp->sockets_per_node, tp->switches_per_socket, tp->gpus_per_switch,
         tp->nics_per_switch, tp->pcie_bytes_per_ns, tp->nic_bytes_per_ns, (tp->flags & 1) != 0};
  if (t.nics != 1) return UNSUPPORTED;   // the rotation model has one NIC per switch
  const int N = t.N(), Q = t.Q();
  auto group = [&](int r) { return r / t.g; };
  auto node = [&](int a) { return a / Q; };
  auto socket = [&](int a) { return (a % Q) / t.switches; };
  // a rational p / q, q > 0
  struct Rat { u128 p, q; };
  auto less = [](const Rat& x, const Rat& y) { return x.p * y.q < y.p * x.q; };
  i64 l = t.pcie;
  { i64 a = t.pcie, b = t.nic; while (b) { i64 r = a % b; a = b; b = r; } l = t.pcie / a * t.nic; }
  u128 total = 0;   // in units of 1 / l ns
  for (int s = 1; s < N; ++s) {
    std::vector<int> src, dst;
    std::vector<std::vector<int>> opts;
    for (int i = 0; i < N; ++i) {
      const int j = (i + s) % N;
      if (D[(size_t)i * N + j] < 0) return INVALID_ARGUMENT;
      if (D[(size_t)i * N + j] == 0) continue;
      const int a = group(i), d = group(j);
      std::vector<int> o;
      if (a == d) o = {PIX};
      else if (node(a) == node(d) && socket(a) == socket(d)) o = nearest ? std::vector<int>{PXB} : std::vector<int>{PXB, NIC};
      else if (node(a) == node(d) && t.sys) o = nearest ? std::vector<int>{SYS} : std::vector<int>{SYS, NIC};
      else o = {NIC};
      src.push_back(i);
      dst.push_back(j);
      opts.push_back(o);
    }
    if (src.empty()) continue;
    const size_t n = src.size();
    std::vector<size_t> odo(n, 0);
    bool have = false;
    Rat best{0, 1};
    while (true) {
      // (kind, index) -> lanes; kind 0 UP, 1 DN (switch), 2 TX, 3 RX (NIC),
      // 4 the socket link (node, source socket, destination socket)
      std::map<std::pair<int, int>, int> share;
      auto xlink = [&](int a, int d) { return (node(a) * t.sockets + socket(a)) * t.sockets + socket(d); };
      for (size_t e = 0; e < n; ++e) {
        const int c = opts[e][odo[e]], a = group(src[e]), d = group(dst[e]);
        if (c == PXB || c == SYS) { share[{0, a}]++; share[{1, d}]++; }
        if (c == SYS) share[{4, xlink(a, d)}]++;
        if (c == NIC) { share[{2, a}]++; share[{3, d}]++; }
      }
      Rat worst{0, 1};
      for (size_t e = 0; e < n; ++e) {
        const int c = opts[e][odo[e]], a = group(src[e]), d = group(dst[e]);
        const u128 x = (u128)D[(size_t)src[e] * N + dst[e]];
        // rate as a fraction cap / sharers; start from the path rate
        Rat rate{(u128)(c == NIC ? std::min(t.pcie, t.nic) : t.pcie), 1};
        auto cap = [&](i64 c2, int k) { Rat r{(u128)c2, (u128)k}; if (less(r, rate)) rate = r; };
        if (c == PXB || c == SYS) { cap(t.pcie, share[{0, a}]); cap(t.pcie, share[{1, d}]); }
        if (c == SYS) cap(t.pcie, share[{4, xlink(a, d)}]);
        if (c == NIC) { cap(t.nic, share[{2, a}]); cap(t.nic, share[{3, d}]); }
        const Rat tm{x * rate.q, rate.p};   // bytes / rate
        if (less(worst, tm)) worst = tm;
      }
      if (!have || less(worst, best)) { best = worst; have = true; }
      size_t e = 0;
      while (e < n && ++odo[e] == opts[e].size()) odo[e++] = 0;
      if (e == n) break;
    }
    // best.p / best.q in units of 1 / l: l * p / q is whole (q divides the rates' lcm times sharers)
    total += (u128)lambda * (u128)l + (u128)l * best.p / best.q;
    if ((u128)l * best.p % best.q != 0) return UNSUPPORTED;   // not on the common grid
  }
  if (total > (u128)INT64_MAX) return UNSUPPORTED;
  *num = (int64_t)total;
  *den = l;
  return OK;
}

// Ulysses head/context re-layout demand: rank j receives its heads of every
// local token, D_self,j = T * heads(j) * head_bytes, D_self,self = 0.
int orc_demand_heads(int64_t T, const int64_t* head_lo, int64_t head_bytes, int32_t N,
                     int32_t self, int64_t* row) {
  if (N < 1 || self < 0 || self >= N) return INVALID_ARGUMENT;
  for (int j = 0; j < N; ++j) row[j] = j == self ? 0 : T * (head_lo[j + 1] - head_lo[j]) * head_bytes;
  return OK;
}

int orc_plan(const orc_catalog* c, const int64_t* D, const orc_params* pp, int32_t k_max,
             int32_t* K, int32_t* fam, int32_t* dst, int32_t* inst, int64_t* bytes,
             int64_t* tau_out, int64_t* trace, int64_t trace_cap, int64_t* trace_n) {
  const Catalog* C = reinterpret_cast<const Catalog*>(c);
  if (!C || !D || !pp || pp->unit_bytes < 1 || pp->k_target < 1 || pp->n_start < 1 ||
      pp->i_aa < 0 || pp->lambda_ns < 0 || k_max < 0)
    return INVALID_ARGUMENT;
  Params P{pp->k_target, pp->lambda_ns, pp->unit_bytes, pp->n_start, pp->i_aa, pp->seed};
  Planner pl(*C, P);
  pl.trace = trace;
  pl.trace_cap = trace ? trace_cap : 0;
  int st = pl.run(D, K, fam, dst, inst, bytes, k_max, tau_out);
  if (trace_n) *trace_n = pl.trace_n;
  return st;
}

// The plan with every evaluated candidate logged, exposed for pinning the
// selection steps: row r of `log` (5 + 3N int64) holds the iteration, the
// family, S, the slowest lane's volume and rate, then for every instance of
// the family in family order its source, destination and volume.
int orc_plan_candidates(const orc_catalog* c, const int64_t* D, const orc_params* pp, int32_t k_max,
                        int32_t* K, int32_t* fam, int32_t* dst, int32_t* inst, int64_t* bytes, int64_t* log,
                        int64_t log_cap, int64_t* log_n) {
  const Catalog* C = reinterpret_cast<const Catalog*>(c);
  if (!C || !D || !pp || !log || pp->unit_bytes < 1 || pp->k_target < 1 || pp->n_start < 1 ||
      pp->i_aa < 0 || pp->lambda_ns < 0 || k_max < 0)
    return INVALID_ARGUMENT;
  Params P{pp->k_target, pp->lambda_ns, pp->unit_bytes, pp->n_start, pp->i_aa, pp->seed};
  Planner pl(*C, P);
  pl.cand_log = log;
  pl.cand_cap = log_cap;
  int st = pl.run(D, K, fam, dst, inst, bytes, k_max, nullptr);
  if (log_n) *log_n = pl.cand_n;
  return st;
}

// Steps 2 and 3 on a given shape m with D as the residual (its quantum as
// at the start of a plan; `iter` keys the random starts), exposed for
// pinning the family choice on any bucket: every candidate is logged as by
// orc_plan_candidates and *chosen receives the family kept.
int orc_shape_candidates(const orc_catalog* c, const int64_t* D, const orc_params* pp, int64_t iter, int32_t m,
                         int64_t* log, int64_t log_cap, int64_t* log_n, int32_t* chosen) {
  const Catalog* C = reinterpret_cast<const Catalog*>(c);
  if (!C || !D || !pp || !log || !chosen || m < 0 || m >= (int32_t)C->shapes.size() || pp->unit_bytes < 1 ||
      pp->k_target < 1 || pp->n_start < 1 || pp->i_aa < 0 || pp->lambda_ns < 0)
    return INVALID_ARGUMENT;
  Params P{pp->k_target, pp->lambda_ns, pp->unit_bytes, pp->n_start, pp->i_aa, pp->seed};
  Planner pl(*C, P);
  if (!pl.load(D)) return INVALID_DEMAND;
  pl.set_quantum();
  pl.K = iter;
  pl.cand_log = log;
  pl.cand_cap = log_cap;
  *chosen = pl.best_candidate(m).f;
  if (log_n) *log_n = pl.cand_n;
  return OK;
}

// One start binding of MultiStartAA before any AA sweep, exposed for
// pinning: D is taken as the residual (its quantum as at the start of a
// plan), `iter` is the iteration number that keys the random starts, start 0
// is the canonical binding with the top credit triple forced in, starts >= 1
// the shuffled ones; both are then made self-transfer free.  src[t], dst[t]:
// the ranks bound to instance t of family f (family order).
int orc_start_binding(const orc_catalog* c, const int64_t* D, const orc_params* pp, int64_t iter, int32_t f,
                      int32_t start, int32_t* src, int32_t* dst) {
  const Catalog* C = reinterpret_cast<const Catalog*>(c);
  if (!C || !D || !pp || f < 0 || f >= (int32_t)C->fams.size() || start < 0 || pp->unit_bytes < 1 ||
      pp->k_target < 1)
    return INVALID_ARGUMENT;
  Params P{pp->k_target, pp->lambda_ns, pp->unit_bytes, pp->n_start, pp->i_aa, pp->seed};
  Planner pl(*C, P);
  if (!pl.load(D)) return INVALID_DEMAND;
  pl.set_quantum();
  pl.K = iter;
  const CFamily& F = C->fams[f];
  std::vector<std::vector<int>> outs, ins;
  pl.group_lists(F, outs, ins);
  Planner::Binding b = start == 0 ? pl.start_forced(F, outs, ins) : pl.start_random(F, f, start, outs, ins);
  for (size_t t = 0; t < F.inst.size(); ++t) {
    src[t] = b.src[t];
    dst[t] = b.dst[t];
  }
  return OK;
}

// The counter-based generator of the random AA starts, exposed for pinning:
// n outputs of SplitMix64 from a raw state, or (when key != 0) from the state
// keyed by (seed, iteration, family, start, group, side) = fields[0..5].
int orc_splitmix_stream(uint64_t state, const uint64_t* fields, int32_t n, uint64_t* out) {
  SplitMix rng{state};
  if (fields) rng = keyed_stream(fields[0], fields[1], fields[2], fields[3], fields[4], fields[5]);
  for (int i = 0; i < n; ++i) out[i] = rng.next();
  return OK;
}

// The planner's exact utility order, exposed for pinning: 1 when the
// candidate (S1, x1, b1) has a strictly larger Eq. (10) utility than
// (S2, x2, b2), where x/b is each candidate's slowest lane.
int orc_utility_greater(int64_t S1, int64_t x1, int64_t b1, int64_t S2, int64_t x2, int64_t b2,
                        int64_t lambda_ns) {
  Catalog dummy;
  dummy.topo = Topo{1, 1, 1, 2, 1, 1, 1};
  dummy.bw_max = 1;
  Params P{1, lambda_ns, 1, 1, 0, 0};
  Planner pl(dummy, P);
  Planner::Eval e1, e2;
  e1.S = S1; e1.xm = x1; e1.bm = b1;
  e2.S = S2; e2.xm = x2; e2.bm = b2;
  return pl.better(e1, e2) ? 1 : 0;
}

// Modeled completion time, Eq. (2), as an exact fraction num / den (ns).
int orc_modeled_time(const orc_catalog* c, int32_t K, int32_t N, const int32_t* inst,
                     const int64_t* bytes, int64_t lambda_ns, int64_t* num, int64_t* den) {
  const Catalog* C = reinterpret_cast<const Catalog*>(c);
  int64_t l = 1;
  for (const auto& r : C->table) {
    int64_t a = l, b = r.bw;
    while (b) { int64_t t = a % b; a = b; b = t; }
    l = l / a * r.bw;
  }
  int64_t total = 0;
  for (int k = 0; k < K; ++k) {
    int64_t worst = 0;
    for (int i = 0; i < N; ++i) {
      int64_t x = bytes[(size_t)k * N + i];
      int64_t bw = C->table[inst[(size_t)k * N + i]].bw;
      worst = std::max(worst, x * (l / bw));
    }
    total += lambda_ns * l + worst;
  }
  *num = total;
  *den = l;
  return OK;
}

// Send-buffer layout (Sec. 5 "Device-resident buffer layout"): for the steps
// in which this rank's lane carries bytes, in schedule order, append the next
// x bytes of the stream to the lane's destination.  Stream j is rank j's
// token rows in (expert, token) order.  step_off[k] is where step k starts.
int orc_pack_rows(const uint8_t* tokens, int64_t T, int64_t row_bytes, const int32_t* sorted_tok,
                  const int64_t* dest_off, int32_t self, int32_t N, int32_t K,
                  const int32_t* dst, const int64_t* bytes, uint8_t* send, int64_t* step_off) {
  std::vector<int64_t> sent(N, 0);
  int64_t o = 0;
  for (int k = 0; k < K; ++k) {
    step_off[k] = o;
    int64_t x = bytes[(size_t)k * N + self];
    int j = dst[(size_t)k * N + self];
    if (x == 0) continue;
    if (x < 0 || x % row_bytes != 0 || j < 0 || j >= N || j == self) return INVALID_ARGUMENT;
    int64_t stream_rows = dest_off[j + 1] - dest_off[j];
    if ((sent[j] + x) / row_bytes > stream_rows) return INVALID_ARGUMENT;
    for (int64_t u = 0; u < x / row_bytes; ++u) {
      int64_t p = dest_off[j] + sent[j] / row_bytes + u;
      int64_t tok = sorted_tok[p];
      if (tok < 0 || tok >= T) return INVALID_ARGUMENT;
      std::memcpy(send + o + u * row_bytes, tokens + tok * row_bytes, (size_t)row_bytes);
    }
    sent[j] += x;
    o += x;
  }
  step_off[K] = o;
  return OK;
}

// Ulysses layout: stream j is, for every local token in order, the bytes of
// the heads rank j owns; units are single heads.
int orc_pack_heads(const uint8_t* act, int64_t T, int64_t token_stride, const int64_t* head_lo,
                   int64_t head_bytes, int32_t self, int32_t N, int32_t K, const int32_t* dst,
                   const int64_t* bytes, uint8_t* send, int64_t* step_off) {
  std::vector<int64_t> sent(N, 0);
  int64_t o = 0;
  for (int k = 0; k < K; ++k) {
    step_off[k] = o;
    int64_t x = bytes[(size_t)k * N + self];
    int j = dst[(size_t)k * N + self];
    if (x == 0) continue;
    if (x < 0 || x % head_bytes != 0 || j < 0 || j >= N || j == self) return INVALID_ARGUMENT;
    int64_t hj = head_lo[j + 1] - head_lo[j];
    if ((sent[j] + x) / head_bytes > T * hj) return INVALID_ARGUMENT;
    for (int64_t u = 0; u < x / head_bytes; ++u) {
      int64_t idx = sent[j] / head_bytes + u;
      int64_t tok = idx / hj, head = head_lo[j] + idx % hj;
      std::memcpy(send + o + u * head_bytes, act + tok * token_stride + head * head_bytes,
                  (size_t)head_bytes);
    }
    sent[j] += x;
    o += x;
  }
  step_off[K] = o;
  return OK;
}

// Buffer layout of a schedule (Sec. 5 "Device-resident buffer layout"), per
// step k and lane i: bytes rank i sent before step k (where the slice starts
// in i's send buffer), bytes i sent to pi_k(i) before step k (where it starts
// in that stream), and bytes pi_k(i) received before step k (where it lands in
// the destination's receive stream, slices in step order).
int orc_layout(int32_t K, int32_t N, const int32_t* dst, const int64_t* bytes, int64_t* send_off,
               int64_t* stream_off, int64_t* recv_off) {
  std::vector<int64_t> sent(N, 0), got(N, 0), pair((size_t)N * N, 0);
  for (int k = 0; k < K; ++k) {
    for (int i = 0; i < N; ++i) {
      const size_t o = (size_t)k * N + i;
      const int j = dst[o];
      if (j < 0 || j >= N) return INVALID_ARGUMENT;
      send_off[o] = sent[i];
      stream_off[o] = pair[(size_t)i * N + j];
      recv_off[o] = got[j];
    }
    for (int i = 0; i < N; ++i) {
      const size_t o = (size_t)k * N + i;
      const int j = dst[o];
      sent[i] += bytes[o];
      pair[(size_t)i * N + j] += bytes[o];
      got[j] += bytes[o];
    }
  }
  return OK;
}

// Receive slots: each token row lands at its own slot of slot_bytes (the row
// rounded up to 128 bytes, Sec. 5 low-latency protocol).  The transfer
// emulation below is test infrastructure: it moves every lane's slice from
// its sender's send buffer (sends: the N buffers back to back, send_base[i]
// where rank i's starts, step_off[i][k] where its step k starts) into rank
// r's receive buffer, slices addressed to r in step order.
int orc_receive(int32_t r, int32_t N, int32_t K, const int32_t* dst, const int64_t* bytes,
                int64_t row_bytes, int64_t slot_bytes, const uint8_t* sends, const int64_t* send_base,
                const int64_t* step_off, uint8_t* recv) {
  int64_t got = 0;
  for (int k = 0; k < K; ++k)
    for (int i = 0; i < N; ++i) {
      const size_t o = (size_t)k * N + i;
      if (dst[o] != r || bytes[o] == 0) continue;
      const int64_t rows = bytes[o] / row_bytes;
      const uint8_t* src = sends + send_base[i] + step_off[(size_t)i * (K + 1) + k];
      for (int64_t u = 0; u < rows; ++u)
        std::memcpy(recv + (got + u) * slot_bytes, src + u * row_bytes, (size_t)row_bytes);
      got += rows;
    }
  return OK;
}

namespace {
// Expert-major output of rank r: local expert e's rows from every source in
// (source rank, token) order.  base[i * eloc + m] is where source i's rows for
// r's m-th local expert start; cum[i * (eloc + 1) + m] where they start in the
// stream from i to r (rows of r's experts in (expert, token) order).
void expert_major(int32_t r, int32_t N, const int32_t* counts, int32_t E, std::vector<int64_t>& base,
                  std::vector<int64_t>& cum) {
  const int eloc = E / N;
  base.assign((size_t)N * eloc, 0);
  cum.assign((size_t)N * (eloc + 1), 0);
  int64_t o = 0;
  for (int m = 0; m < eloc; ++m)
    for (int i = 0; i < N; ++i) {
      base[(size_t)i * eloc + m] = o;
      o += counts[(size_t)i * E + r * eloc + m];
    }
  for (int i = 0; i < N; ++i)
    for (int m = 0; m < eloc; ++m)
      cum[(size_t)i * (eloc + 1) + m + 1] = cum[(size_t)i * (eloc + 1) + m] + counts[(size_t)i * E + r * eloc + m];
}

// Output row of stream row q from source i.
int64_t out_row(const std::vector<int64_t>& base, const std::vector<int64_t>& cum, int eloc, int i, int64_t q) {
  int m = 0;
  while (m + 1 < eloc && q >= cum[(size_t)i * (eloc + 1) + m + 1]) ++m;
  return base[(size_t)i * eloc + m] + (q - cum[(size_t)i * (eloc + 1) + m]);
}
}  // namespace

// Dispatch receive (Sec. 5: the receive kernel unpacks straight into the
// output layout): rank r's receive buffer, slices in step order, into the
// expert-major output (slots of slot_bytes).  counts: [N, E] assignments per
// (source rank, expert).
int orc_unpack_rows(const uint8_t* recv, int32_t r, int32_t N, int32_t K, const int32_t* dst,
                    const int64_t* bytes, int64_t row_bytes, int64_t slot_bytes, const int32_t* counts,
                    int32_t E, uint8_t* out) {
  if (E % N != 0) return INVALID_ARGUMENT;
  std::vector<int64_t> base, cum;
  expert_major(r, N, counts, E, base, cum);
  std::vector<int64_t> sent(N, 0);
  int64_t got = 0;
  for (int k = 0; k < K; ++k)
    for (int i = 0; i < N; ++i) {
      const size_t o = (size_t)k * N + i;
      if (dst[o] != r || bytes[o] == 0) continue;
      const int64_t rows = bytes[o] / row_bytes;
      for (int64_t u = 0; u < rows; ++u) {
        const int64_t q = sent[i] + u;
        if (q >= cum[(size_t)i * (E / N + 1) + E / N]) return INVALID_ARGUMENT;
        std::memcpy(out + out_row(base, cum, E / N, i, q) * slot_bytes, recv + (got + u) * slot_bytes,
                    (size_t)row_bytes);
      }
      sent[i] += rows;
      got += rows;
    }
  return OK;
}

// Combine send (the return AlltoAllv, planned on the transposed demand):
// stream r -> i is rank r's expert-major rows from source i in (expert,
// token) order; lane r's steps append its next slice in schedule order.
int orc_pack_combine(const uint8_t* out, int32_t r, int32_t N, int32_t K, const int32_t* dst,
                     const int64_t* bytes, int64_t row_bytes, int64_t slot_bytes, const int32_t* counts,
                     int32_t E, uint8_t* send, int64_t* step_off) {
  if (E % N != 0) return INVALID_ARGUMENT;
  std::vector<int64_t> base, cum;
  expert_major(r, N, counts, E, base, cum);
  std::vector<int64_t> sent(N, 0);
  int64_t o = 0;
  for (int k = 0; k < K; ++k) {
    step_off[k] = o;
    const size_t x = (size_t)k * N + r;
    const int i = dst[x];
    if (bytes[x] == 0) continue;
    if (i < 0 || i >= N || i == r || bytes[x] % row_bytes != 0) return INVALID_ARGUMENT;
    const int64_t rows = bytes[x] / row_bytes;
    for (int64_t u = 0; u < rows; ++u) {
      const int64_t q = sent[i] + u;
      if (q >= cum[(size_t)i * (E / N + 1) + E / N]) return INVALID_ARGUMENT;
      std::memcpy(send + o + u * row_bytes, out + out_row(base, cum, E / N, i, q) * slot_bytes, (size_t)row_bytes);
    }
    sent[i] += rows;
    o += bytes[x];
  }
  step_off[K] = o;
  return OK;
}

// Combine receive at source rank i: the stream from r carries the rows of
// i's assignments to r's experts in (expert, token) order, i.e. i's sorted
// list for destination r; each row goes to its (token, routing slot) slot of
// combined [T, k].
int orc_unpack_combine(const uint8_t* recv, int32_t self, int32_t N, int32_t K, const int32_t* dst,
                       const int64_t* bytes, int64_t row_bytes, int64_t slot_bytes, int64_t T, int32_t k,
                       const int32_t* sorted_tok, const uint8_t* sorted_slot, const int64_t* dest_off,
                       uint8_t* combined) {
  std::vector<int64_t> sent(N, 0);
  int64_t got = 0;
  for (int kk = 0; kk < K; ++kk)
    for (int r = 0; r < N; ++r) {
      const size_t o = (size_t)kk * N + r;
      if (dst[o] != self || bytes[o] == 0) continue;
      const int64_t rows = bytes[o] / row_bytes;
      for (int64_t u = 0; u < rows; ++u) {
        const int64_t p = dest_off[r] + sent[r] + u;
        if (p >= dest_off[r + 1]) return INVALID_ARGUMENT;
        const int64_t t = sorted_tok[p];
        const int c = sorted_slot[p];
        if (t < 0 || t >= T || c >= k) return INVALID_ARGUMENT;
        std::memcpy(combined + (t * k + c) * slot_bytes, recv + (got + u) * slot_bytes, (size_t)row_bytes);
      }
      sent[r] += rows;
      got += rows;
    }
  return OK;
}

}  // extern "C"
