// Modeled completion time of a fixed cyclic peer rotation, the baseline of
// the peer/path ablation (Sec. 6.3, Table 3: "fixed peer rotation").
//
// Stage s = 1 .. N-1 pairs rank i with rank (i + s) mod N and moves the whole
// D_i,(i+s) at once; a stage whose lanes carry nothing is skipped.  A lane's
// path is its pair's nearest one (PIX in a switch, PXB between two switches
// of a socket, SYS between sockets when enabled, the NICs otherwise) or, with
// dynamic paths, whichever of the pair's paths makes the stage finish first.
// Unlike a catalog channel, a rotation stage may put several lanes on one
// directed resource (a switch's uplink or downlink, a socket link, a NIC's
// transmit or receive side): those lanes share
// it equally, so a lane runs at min(path rate, capacity / lanes) over its
// resources.  A stage takes lambda plus its slowest lane's bytes / rate.
// Everything is exact: times are kept over the common denominator of the
// rates.
#include <algorithm>
#include <vector>

#include "internal.h"

namespace vp {
namespace {

struct Lane {
  int64_t x;
  int a, d;            // source and destination group
  int opt[2], nopt;    // candidate path classes
};

int64_t gcd64(int64_t a, int64_t b) {
  while (b) {
    int64_t t = a % b;
    a = b;
    b = t;
  }
  return a;
}

}  // namespace

vp_status rotation_time(const vp_catalog& c, const int64_t* D, int rule, int64_t lambda, int64_t* num,
                        int64_t* den) {
  if (c.topo.nics_per_switch != 1)
    return set_error(VP_ERR_UNSUPPORTED, "the rotation model takes one NIC per switch");
  const int N = c.N, g = c.g, Q = c.Q, G = c.G;
  const int W = c.topo.switches_per_socket, S = c.topo.sockets_per_node;
  const bool sys = (c.topo.flags & VP_TOPO_SYS_P2P) != 0;
  const int64_t pcie = c.topo.pcie_bytes_per_ns, nic = c.topo.nic_bytes_per_ns;
  const int64_t nic_path = std::min(pcie, nic);
  const int64_t l = pcie / gcd64(pcie, nic) * nic;   // common denominator of every rate below
  __int128 total = 0;
  std::vector<Lane> lanes;
  std::vector<int> up(G), dn(G), tx(G), rx(G), xs(c.nn * S * S);
  auto xlink = [&](int a, int d) { return ((a / Q) * S + (a % Q) / W) * S + (d % Q) / W; };
  for (int s = 1; s < N; ++s) {
    lanes.clear();
    for (int i = 0; i < N; ++i) {
      const int j = (i + s) % N;
      const int64_t x = D[(size_t)i * N + j];
      if (x == 0) continue;
      Lane ln{x, i / g, j / g, {VP_PATH_PIX, VP_PATH_PIX}, 1};
      const bool same_node = ln.a / Q == ln.d / Q;
      const bool same_socket = same_node && (ln.a % Q) / W == (ln.d % Q) / W;
      if (ln.a == ln.d) {
        ln.opt[0] = VP_PATH_PIX;
      } else if (same_socket || (same_node && sys)) {
        ln.opt[0] = same_socket ? VP_PATH_PXB : VP_PATH_SYS;   // nearest
        ln.opt[1] = VP_PATH_NIC;
        ln.nopt = rule == 1 ? 1 : 2;
      } else {
        ln.opt[0] = VP_PATH_NIC;
      }
      lanes.push_back(ln);
    }
    if (lanes.empty()) continue;
    std::vector<int> var;
    for (size_t t = 0; t < lanes.size(); ++t)
      if (lanes[t].nopt == 2) var.push_back((int)t);
    if (var.size() > 20) return set_error(VP_ERR_UNSUPPORTED, "more than 20 lanes with a path choice in a stage");
    __int128 best = -1;
    std::vector<int> pick(lanes.size());
    for (uint32_t mask = 0; mask < (1u << var.size()); ++mask) {
      for (size_t t = 0; t < lanes.size(); ++t) pick[t] = lanes[t].opt[0];
      for (size_t v = 0; v < var.size(); ++v)
        if (mask >> v & 1) pick[var[v]] = lanes[var[v]].opt[1];
      std::fill(up.begin(), up.end(), 0);
      std::fill(dn.begin(), dn.end(), 0);
      std::fill(tx.begin(), tx.end(), 0);
      std::fill(rx.begin(), rx.end(), 0);
      std::fill(xs.begin(), xs.end(), 0);
      for (size_t t = 0; t < lanes.size(); ++t) {
        if (pick[t] == VP_PATH_PXB || pick[t] == VP_PATH_SYS) { up[lanes[t].a]++; dn[lanes[t].d]++; }
        if (pick[t] == VP_PATH_SYS) xs[xlink(lanes[t].a, lanes[t].d)]++;
        if (pick[t] == VP_PATH_NIC) { tx[lanes[t].a]++; rx[lanes[t].d]++; }
      }
      // slowest lane: bytes * (l / rate), the rate being the path's or a share
      __int128 worst = 0;
      for (size_t t = 0; t < lanes.size(); ++t) {
        const Lane& ln = lanes[t];
        __int128 per = 0;   // l / rate
        if (pick[t] == VP_PATH_PIX) {
          per = l / pcie;
        } else if (pick[t] == VP_PATH_PXB) {
          per = std::max<__int128>(l / pcie, (__int128)std::max(up[ln.a], dn[ln.d]) * (l / pcie));
        } else if (pick[t] == VP_PATH_SYS) {
          const int sh = std::max(std::max(up[ln.a], dn[ln.d]), xs[xlink(ln.a, ln.d)]);
          per = std::max<__int128>(l / pcie, (__int128)sh * (l / pcie));
        } else {
          per = std::max<__int128>(l / nic_path, (__int128)std::max(tx[ln.a], rx[ln.d]) * (l / nic));
        }
        worst = std::max(worst, (__int128)ln.x * per);
      }
      if (best < 0 || worst < best) best = worst;
    }
    total += (__int128)lambda * l + best;
  }
  if (total > (__int128)INT64_MAX) return set_error(VP_ERR_UNSUPPORTED, "modeled time overflows");
  *num = (int64_t)total;
  *den = l;
  return VP_OK;
}

}  // namespace vp
