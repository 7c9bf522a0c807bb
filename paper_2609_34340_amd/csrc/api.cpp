// C-ABI entry points: argument checks, error reporting, catalog handles.
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstring>
#include <exception>
#include <new>

#include "internal.h"

namespace vp {

namespace {
thread_local std::string g_last_error;
}

vp_status set_error(vp_status s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

}  // namespace vp

using vp::set_error;

extern "C" {

const char* vp_status_string(vp_status s) {
  switch (s) {
    case VP_OK: return "ok";
    case VP_ERR_INVALID_ARGUMENT: return "invalid argument";
    case VP_ERR_INVALID_DEMAND: return "invalid demand";
    case VP_ERR_NO_PROGRESS: return "no progress";
    case VP_ERR_CAPACITY: return "capacity exceeded";
    case VP_ERR_UNSUPPORTED: return "unsupported";
    case VP_ERR_HIP: return "HIP error";
  }
  return "unknown status";
}

const char* vp_last_error(void) { return vp::g_last_error.c_str(); }

}  // extern "C"

namespace {

vp_status check_topology(const vp_topology& t) {
  if ((t.flags & ~VP_TOPO_SYS_P2P) != 0) return set_error(VP_ERR_UNSUPPORTED, "unknown topology flags");
  if ((t.flags & VP_TOPO_SYS_P2P) && t.sockets_per_node > 4)
    return set_error(VP_ERR_UNSUPPORTED, "cross-socket peer to peer needs at most 4 sockets");
  if (t.n_nodes < 1 || t.n_nodes > vp::kMaxNodes)
    return set_error(VP_ERR_UNSUPPORTED, "n_nodes must be in [1, 256]");
  if (t.sockets_per_node < 1 || t.switches_per_socket < 1 ||
      t.sockets_per_node * t.switches_per_socket > vp::kMaxSlotsPerNode)
    return set_error(VP_ERR_UNSUPPORTED, "sockets*switches per node must be in [1, 8]");
  if (t.gpus_per_switch < 2 || t.gpus_per_switch > vp::kMaxGpusPerSwitch)
    return set_error(VP_ERR_UNSUPPORTED, "gpus_per_switch must be in [2, 4]");
  if (t.nics_per_switch < 1 || t.nics_per_switch > 4)
    return set_error(VP_ERR_UNSUPPORTED, "nics_per_switch must be in [1, 4]");
  {
    // one bit per directed resource of a node (UP, DN per switch; TX, RX per
    // NIC; socket links) and node-local instance ids below 256
    const int64_t S = t.sockets_per_node, W = t.switches_per_socket, Q = S * W, m = t.nics_per_switch;
    const bool sys = (t.flags & VP_TOPO_SYS_P2P) != 0;
    if (2 * Q + 2 * Q * m + (sys ? S * S : 0) > 64)
      return set_error(VP_ERR_UNSUPPORTED, "too many switches and NICs per node (resource bits)");
    const int64_t n_inst = Q * t.gpus_per_switch + S * W * (W - 1) + Q * Q * m * m + (sys ? Q * Q - S * W * W : 0);
    if (n_inst > 256) return set_error(VP_ERR_UNSUPPORTED, "more than 256 node-local path instances");
  }
  if (t.pcie_bytes_per_ns < 1 || t.nic_bytes_per_ns < 1)
    return set_error(VP_ERR_INVALID_ARGUMENT, "rates must be positive");
  int64_t N = (int64_t)t.n_nodes * t.sockets_per_node * t.switches_per_socket * t.gpus_per_switch;
  if (N > vp::kMaxRanks) return set_error(VP_ERR_UNSUPPORTED, "more than 1024 ranks");
  return VP_OK;
}

}  // namespace

extern "C" {

vp_status vp_build_catalog(const vp_topology* t, vp_catalog** out) {
  if (!t || !out) return set_error(VP_ERR_INVALID_ARGUMENT, "null topology or output");
  *out = nullptr;
  vp_status s = check_topology(*t);
  if (s != VP_OK) return s;
  vp_catalog* c = new (std::nothrow) vp_catalog();
  if (!c) return set_error(VP_ERR_INVALID_ARGUMENT, "out of host memory");
  try {
    s = vp::build_catalog_host(*t, *c);
  } catch (const std::bad_alloc&) {
    s = set_error(VP_ERR_UNSUPPORTED, "out of host memory while building the catalog");
  } catch (const std::exception& e) {
    s = set_error(VP_ERR_UNSUPPORTED, std::string("catalog build failed: ") + e.what());
  }
  if (s != VP_OK) {
    delete c;
    return s;
  }
  *out = c;
  return VP_OK;
}

vp_status vp_catalog_restrict(const vp_catalog* c, int32_t rule, vp_catalog** out) {
  if (!c || !out) return set_error(VP_ERR_INVALID_ARGUMENT, "null catalog or output");
  *out = nullptr;
  vp_catalog* r = new (std::nothrow) vp_catalog();
  if (!r) return set_error(VP_ERR_INVALID_ARGUMENT, "out of host memory");
  vp_status s = vp::restrict_catalog(*c, rule, *r);
  if (s != VP_OK) {
    delete r;
    return s;
  }
  *out = r;
  return VP_OK;
}

vp_status vp_catalog_save(const vp_catalog* c, void* buf, size_t capacity, size_t* size) {
  if (!c || !size) return set_error(VP_ERR_INVALID_ARGUMENT, "null catalog or size");
  const std::vector<uint8_t> b = vp::serialize_catalog(*c);
  *size = b.size();
  if (!buf) return VP_OK;
  if (capacity < b.size()) return set_error(VP_ERR_CAPACITY, "buffer smaller than the serialized catalog");
  std::memcpy(buf, b.data(), b.size());
  return VP_OK;
}

vp_status vp_catalog_load(const void* buf, size_t size, vp_catalog** out) {
  if (!buf || !out) return set_error(VP_ERR_INVALID_ARGUMENT, "null buffer or output");
  *out = nullptr;
  vp_catalog* c = new (std::nothrow) vp_catalog();
  if (!c) return set_error(VP_ERR_INVALID_ARGUMENT, "out of host memory");
  vp_status s = vp::deserialize_catalog((const uint8_t*)buf, size, *c, check_topology);
  if (s != VP_OK) {
    delete c;
    return s;
  }
  *out = c;
  return VP_OK;
}

vp_status vp_catalog_info(const vp_catalog* c, int64_t info[8]) {
  if (!c || !info) return set_error(VP_ERR_INVALID_ARGUMENT, "null catalog or info");
  info[0] = c->N;
  info[1] = c->G;
  info[2] = c->g;
  info[3] = c->Q;
  info[4] = c->nn;
  info[5] = c->lay.J;
  info[6] = c->lay.F;
  info[7] = (int64_t)c->icls.size();
  return VP_OK;
}

vp_status vp_catalog_instances(const vp_catalog* c, int32_t* cls, int32_t* src, int32_t* dst,
                               int32_t* copy, int64_t* bw) {
  if (!c || !cls || !src || !dst || !copy || !bw)
    return set_error(VP_ERR_INVALID_ARGUMENT, "null argument");
  for (size_t i = 0; i < c->icls.size(); ++i) {
    cls[i] = c->icls[i]; src[i] = c->isrc[i]; dst[i] = c->idst[i]; copy[i] = c->icopy[i]; bw[i] = c->ibw[i];
  }
  return VP_OK;
}

vp_status vp_catalog_shapes(const vp_catalog* c, int32_t* k, int32_t* fam_begin, int32_t* fam_end,
                            int32_t* L, int32_t* R) {
  if (!c || !k || !fam_begin || !fam_end || !L || !R)
    return set_error(VP_ERR_INVALID_ARGUMENT, "null argument");
  const int QQ = c->Q * c->Q;
  int64_t j = 0;
  for (int s = 0; s < c->nn; ++s) {
    int pb = s == 0 ? 0 : c->J0, pe = s == 0 ? c->J0 : c->J0 + c->J1;
    for (int p = pb; p < pe; ++p, ++j) {
      k[j] = s;
      int64_t base = s == 0 ? 0 : (int64_t)c->F0 + (int64_t)(s - 1) * c->F1 - c->F0;
      fam_begin[j] = (int32_t)(c->pat_fb[p] + base);
      fam_end[j] = (int32_t)(c->pat_fe[p] + base);
      std::memcpy(L + j * QQ, c->patL[p].data(), QQ * sizeof(int32_t));
      std::memcpy(R + j * QQ, c->patR[p].data(), QQ * sizeof(int32_t));
    }
  }
  return VP_OK;
}

vp_status vp_catalog_families(const vp_catalog* c, int32_t* shape, int32_t* k, int32_t* ids) {
  if (!c || !shape || !k || !ids) return set_error(VP_ERR_INVALID_ARGUMENT, "null argument");
  const int QG = c->Q * c->g;
  std::vector<int32_t> pat_of(c->F0 + c->F1, 0);
  for (int p = 0; p < c->J0 + c->J1; ++p)
    for (int f = c->pat_fb[p]; f < c->pat_fe[p]; ++f) pat_of[f] = p;
  int64_t f = 0;
  for (int s = 0; s < c->nn; ++s) {
    int lb = s == 0 ? 0 : c->F0, le = s == 0 ? c->F0 : c->F0 + c->F1;
    for (int lf = lb; lf < le; ++lf, ++f) {
      k[f] = s;
      int p = pat_of[lf];
      shape[f] = s == 0 ? p : (int32_t)(c->J0 + (int64_t)(s - 1) * c->J1 + (p - c->J0));
      std::memcpy(ids + f * QG, c->lfam[lf].data(), QG * sizeof(int32_t));
    }
  }
  return VP_OK;
}

vp_status vp_catalog_upload(vp_catalog* c, void* stream) {
  if (!c) return set_error(VP_ERR_INVALID_ARGUMENT, "null catalog");
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return set_error(VP_ERR_HIP, "hipGetDevice failed");
  if (c->dev && c->dev_id == dev) return VP_OK;
  if (c->dev) {
    (void)hipFree(c->dev);
    c->dev = nullptr;
  }
  size_t bytes = c->image.size() * sizeof(int32_t);
  if (hipMalloc(&c->dev, bytes) != hipSuccess) return set_error(VP_ERR_HIP, "hipMalloc of catalog failed");
  hipStream_t s = (hipStream_t)stream;
  if (hipMemcpyAsync(c->dev, c->image.data(), bytes, hipMemcpyHostToDevice, s) != hipSuccess ||
      hipStreamSynchronize(s) != hipSuccess) {
    (void)hipFree(c->dev);
    c->dev = nullptr;
    return set_error(VP_ERR_HIP, "catalog upload failed");
  }
  c->dev_id = dev;
  return VP_OK;
}

void vp_catalog_free(vp_catalog* c) {
  if (!c) return;
  if (c->dev) (void)hipFree(c->dev);
  delete c;
}

size_t vp_demand_workspace(int32_t R, int64_t T, int32_t k, int32_t E) {
  if (R < 1 || T < 0 || k < 1 || E < 1) return 0;
  return vp::demand_workspace(R, T, k, E);
}

vp_status vp_demand(const int32_t* routing, int32_t R, int64_t T, int32_t k, int32_t E,
                    int32_t n_ranks, int32_t first_rank, int32_t sort_row, int64_t unit_bytes,
                    int32_t* counts, int64_t* demand, int32_t* sorted_tok, uint8_t* sorted_slot,
                    int64_t* dest_off, int32_t* dev_status, void* ws, size_t ws_bytes, void* stream) {
  if (R < 1 || T < 0 || k < 1 || k > 255 || E < 1 || n_ranks < 1 || E % n_ranks != 0 || E > 4096)
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad demand sizes (E a multiple of N, <= 4096; k <= 255)");
  if (T * (int64_t)k >= (int64_t(1) << 31)) return set_error(VP_ERR_UNSUPPORTED, "T*k must be < 2^31");
  if (first_rank < 0 || first_rank + R > n_ranks) return set_error(VP_ERR_INVALID_ARGUMENT, "rank range");
  if (sort_row < -1 || sort_row >= R) return set_error(VP_ERR_INVALID_ARGUMENT, "sort_row");
  if (unit_bytes < 1) return set_error(VP_ERR_INVALID_ARGUMENT, "unit_bytes");
  if ((T > 0 && !routing) || !counts || !demand || !dev_status)
    return set_error(VP_ERR_INVALID_ARGUMENT, "null pointer");
  if (sort_row >= 0 && ((T > 0 && !sorted_tok) || !dest_off))
    return set_error(VP_ERR_INVALID_ARGUMENT, "null sort output");
  if (ws_bytes < vp::demand_workspace(R, T, k, E) || !ws)
    return set_error(VP_ERR_INVALID_ARGUMENT, "workspace too small");
  vp::DemandLaunch a{routing, R, T, k, E, n_ranks, first_rank, sort_row, unit_bytes, counts, demand,
                     sorted_tok, sorted_slot, dest_off, dev_status, ws, ws_bytes};
  return vp::launch_demand(a, stream);
}

vp_status vp_demand_heads(int64_t T, const int64_t* head_lo, int64_t head_bytes, int32_t n_ranks,
                          int32_t first_rank, int32_t R, int64_t* demand, int32_t* dev_status,
                          void* stream) {
  if (T < 0 || !head_lo || head_bytes < 1 || n_ranks < 1 || n_ranks > vp::kMaxRanks || R < 1 ||
      first_rank < 0 || first_rank + R > n_ranks || !demand || !dev_status)
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad head-demand arguments");
  return vp::launch_demand_heads(T, head_lo, head_bytes, n_ranks, first_rank, R, demand, dev_status, stream);
}

vp_status vp_control_words(const int32_t* counts, int32_t R, int32_t E, int32_t n_ranks, int32_t first_rank,
                           uint32_t* words, int32_t* dev_status, void* stream) {
  if (!counts || !words || !dev_status || R < 0 || n_ranks < 1 || n_ranks > vp::kMaxRanks || E < n_ranks ||
      E % n_ranks != 0 || first_rank < 0 || first_rank + R > n_ranks)
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad control-word arguments");
  if (E / n_ranks > 31) return set_error(VP_ERR_UNSUPPORTED, "more than 31 local experts per rank");
  return vp::launch_control_words(counts, R, E, n_ranks, first_rank, words, dev_status, stream);
}

vp_status vp_receive_counts(const uint32_t* words, int64_t word_stride, const int32_t* signal, int32_t n_ranks,
                            int32_t n_local, int32_t* counts, void* stream) {
  if (!words || !signal || !counts || word_stride < 1 || n_ranks < 1 || n_ranks > vp::kMaxRanks || n_local < 1)
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad receive-count arguments");
  if (n_local > 31) return set_error(VP_ERR_UNSUPPORTED, "more than 31 local experts per rank");
  return vp::launch_receive_counts(words, word_stride, signal, n_ranks, n_local, counts, stream);
}

void vp_plan_params_default(int32_t n_ranks, int64_t unit_bytes, vp_plan_params* p) {
  if (!p) return;
  p->k_target = 2 * (int64_t)n_ranks;
  p->lambda_ns = 10000;
  p->unit_bytes = unit_bytes;
  p->n_start = 4;
  p->i_aa = 8;
  p->seed = 0;
  p->k_max = 8 * n_ranks;
  p->reserved = 0;
}

size_t vp_plan_workspace(const vp_catalog* c, const vp_plan_params* p) { return vp_plan_batch_workspace(c, p, 1); }

size_t vp_plan_batch_workspace(const vp_catalog* c, const vp_plan_params* p, int32_t batch) {
  (void)p;
  if (!c || batch < 1) return 0;
  return (size_t)batch * (size_t)c->N * (size_t)c->N * sizeof(int64_t);
}

vp_status vp_plan_batch(const vp_catalog* c, int32_t batch, const int64_t* demand, const vp_plan_params* p,
                        int32_t* K, int32_t* family, int32_t* dst, int32_t* inst, int64_t* bytes, int64_t* send_off,
                        int64_t* stream_off, int32_t* recv_src, int64_t* tau, int32_t* dev_status, void* ws,
                        size_t ws_bytes, void* stream) {
  if (!c || !demand || !p || !K || !family || !dst || !inst || !bytes || !dev_status)
    return set_error(VP_ERR_INVALID_ARGUMENT, "null pointer");
  if (batch < 1 || batch > 65535) return set_error(VP_ERR_INVALID_ARGUMENT, "batch must be in [1, 65535]");
  if ((send_off == nullptr) != (stream_off == nullptr))
    return set_error(VP_ERR_INVALID_ARGUMENT, "send_off and stream_off go together");
  if (!c->dev) return set_error(VP_ERR_INVALID_ARGUMENT, "catalog not uploaded");
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev != c->dev_id)
    return set_error(VP_ERR_INVALID_ARGUMENT, "catalog uploaded to another device");
  if (p->k_target < 1 || p->lambda_ns < 0 || p->unit_bytes < 1 || p->n_start < 1 ||
      p->n_start > vp::kMaxStarts || p->i_aa < 0 || p->k_max < 1)
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad plan parameters");
  if (p->lambda_ns > (int64_t(1) << 40) || p->k_target > (int64_t(1) << 40))
    return set_error(VP_ERR_UNSUPPORTED, "lambda or k_target too large");
  if (ws_bytes < vp_plan_batch_workspace(c, p, batch) || !ws)
    return set_error(VP_ERR_INVALID_ARGUMENT, "workspace too small");
  vp::PlanLaunch a{c, demand, (int64_t*)ws, *p, K, family, dst, inst, bytes, tau, send_off, stream_off, recv_src,
                   dev_status, batch};
  return vp::launch_plan(a, stream);
}

vp_status vp_plan(const vp_catalog* c, const int64_t* demand, const vp_plan_params* p, int32_t* K,
                  int32_t* family, int32_t* dst, int32_t* inst, int64_t* bytes, int64_t* send_off,
                  int64_t* stream_off, int32_t* recv_src, int64_t* tau, int32_t* dev_status, void* ws,
                  size_t ws_bytes, void* stream) {
  return vp_plan_batch(c, 1, demand, p, K, family, dst, inst, bytes, send_off, stream_off, recv_src, tau,
                       dev_status, ws, ws_bytes, stream);
}

vp_status vp_plan_noalloc(const vp_catalog* c, const int64_t* demand, const vp_plan_params* p, int32_t* K,
                          int32_t* family, int32_t* dst, int32_t* inst, int64_t* bytes, int64_t* send_off,
                          int64_t* stream_off, int32_t* recv_src, int64_t* tau, int32_t* dev_status, void* stream) {
  if (!c) return set_error(VP_ERR_INVALID_ARGUMENT, "null catalog");
  void* residual = nullptr;
  const vp_status st = vp::static_residual(c->N, &residual);
  if (st != VP_OK) return st;
  return vp_plan_batch(c, 1, demand, p, K, family, dst, inst, bytes, send_off, stream_off, recv_src, tau,
                       dev_status, residual, (size_t)c->N * (size_t)c->N * sizeof(int64_t), stream);
}

size_t vp_pack_workspace(int32_t k_max, int64_t send_capacity, int64_t unit_bytes, int64_t T, int32_t k) {
  if (k_max < 1 || send_capacity < 0 || unit_bytes < 1 || T < 0 || k < 0) return 0;
  return vp::pack_workspace(k_max, send_capacity, unit_bytes, T, k);
}

namespace {

vp_status pack_rows_stages(int stages, const void* tokens, int64_t T, int32_t k, int64_t row_bytes,
                           const int32_t* sorted_tok, const uint8_t* sorted_slot, const int64_t* dest_off,
                           int32_t self_rank,
                           int32_t n_ranks, const int32_t* K, const int32_t* dst, const int64_t* bytes,
                           const int64_t* send_off, const int64_t* stream_off, int32_t k_max, void* send,
                           int64_t send_capacity, int64_t* step_off, int32_t* dev_status, void* ws,
                           size_t ws_bytes, void* stream) {
  if ((send_off == nullptr) != (stream_off == nullptr))
    return set_error(VP_ERR_INVALID_ARGUMENT, "send_off and stream_off go together");
  if (T < 0 || k < 1 || row_bytes < 16 || row_bytes % 16 != 0 || n_ranks < 1 || n_ranks > vp::kMaxRanks ||
      self_rank < 0 || self_rank >= n_ranks || k_max < 1 || send_capacity < 0)
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad pack sizes (row_bytes must be a multiple of 16)");
  if (!dest_off || !K || !dst || !bytes || !step_off || !dev_status ||
      (T > 0 && (!tokens || !sorted_tok || !sorted_slot)) ||
      ((stages & 2) && send_capacity > 0 && !send))
    return set_error(VP_ERR_INVALID_ARGUMENT, "null pointer");
  if (ws_bytes < vp::pack_workspace(k_max, send_capacity, row_bytes, T, k) || !ws)
    return set_error(VP_ERR_INVALID_ARGUMENT, "workspace too small");
  vp::PackLaunch a{0, stages, tokens, T, k, row_bytes, row_bytes, sorted_tok, sorted_slot, dest_off, nullptr,
                   self_rank, n_ranks,
                   K, dst, bytes, send_off, stream_off, k_max, send, send_capacity, step_off, dev_status, ws,
                   ws_bytes};
  return vp::launch_pack(a, stream);
}

vp_status pack_heads_stages(int stages, const void* act, int64_t T, int64_t token_stride,
                            const int64_t* head_lo, int64_t head_bytes, int32_t self_rank, int32_t n_ranks,
                            const int32_t* K, const int32_t* dst, const int64_t* bytes,
                            const int64_t* send_off, const int64_t* stream_off, int32_t k_max, void* send,
                            int64_t send_capacity, int64_t* step_off, int32_t* dev_status, void* ws,
                            size_t ws_bytes, void* stream) {
  if ((send_off == nullptr) != (stream_off == nullptr))
    return set_error(VP_ERR_INVALID_ARGUMENT, "send_off and stream_off go together");
  if (T < 0 || head_bytes < 16 || head_bytes % 16 != 0 || token_stride < head_bytes ||
      token_stride % 16 != 0 || n_ranks < 1 || n_ranks > vp::kMaxRanks || self_rank < 0 ||
      self_rank >= n_ranks || k_max < 1 || send_capacity < 0)
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad pack sizes (head_bytes and stride multiples of 16)");
  if (!head_lo || !K || !dst || !bytes || !step_off || !dev_status || (T > 0 && !act) ||
      ((stages & 2) && send_capacity > 0 && !send))
    return set_error(VP_ERR_INVALID_ARGUMENT, "null pointer");
  if (ws_bytes < vp::pack_workspace(k_max, send_capacity, head_bytes, T, 0) || !ws)
    return set_error(VP_ERR_INVALID_ARGUMENT, "workspace too small");
  vp::PackLaunch a{1, stages, act, T, 0, head_bytes, token_stride, nullptr, nullptr, nullptr, head_lo,
                   self_rank, n_ranks,
                   K, dst, bytes, send_off, stream_off, k_max, send, send_capacity, step_off, dev_status, ws,
                   ws_bytes};
  return vp::launch_pack(a, stream);
}

}  // namespace

vp_status vp_pack_rows(const void* tokens, int64_t T, int32_t k, int64_t row_bytes, const int32_t* sorted_tok,
                       const uint8_t* sorted_slot, const int64_t* dest_off, int32_t self_rank, int32_t n_ranks,
                       const int32_t* K, const int32_t* dst, const int64_t* bytes, const int64_t* send_off,
                       const int64_t* stream_off, int32_t k_max, void* send, int64_t send_capacity,
                       int64_t* step_off, int32_t* dev_status, void* ws, size_t ws_bytes, void* stream) {
  return pack_rows_stages(3, tokens, T, k, row_bytes, sorted_tok, sorted_slot, dest_off, self_rank, n_ranks, K,
                          dst, bytes,
                          send_off, stream_off, k_max, send, send_capacity, step_off, dev_status, ws, ws_bytes,
                          stream);
}

vp_status vp_pack_prepare_rows(const void* tokens, int64_t T, int32_t k, int64_t row_bytes,
                               const int32_t* sorted_tok, const uint8_t* sorted_slot,
                               const int64_t* dest_off, int32_t self_rank, int32_t n_ranks,
                               const int32_t* K, const int32_t* dst, const int64_t* bytes,
                               const int64_t* send_off, const int64_t* stream_off, int32_t k_max,
                               int64_t send_capacity, int64_t* step_off, int32_t* dev_status, void* ws,
                               size_t ws_bytes, void* stream) {
  return pack_rows_stages(1, tokens, T, k, row_bytes, sorted_tok, sorted_slot, dest_off, self_rank, n_ranks, K,
                          dst, bytes,
                          send_off, stream_off, k_max, nullptr, send_capacity, step_off, dev_status, ws,
                          ws_bytes, stream);
}

vp_status vp_pack_heads(const void* act, int64_t T, int64_t token_stride, const int64_t* head_lo,
                        int64_t head_bytes, int32_t self_rank, int32_t n_ranks, const int32_t* K,
                        const int32_t* dst, const int64_t* bytes, const int64_t* send_off,
                        const int64_t* stream_off, int32_t k_max, void* send, int64_t send_capacity,
                        int64_t* step_off, int32_t* dev_status, void* ws, size_t ws_bytes, void* stream) {
  return pack_heads_stages(3, act, T, token_stride, head_lo, head_bytes, self_rank, n_ranks, K, dst, bytes,
                           send_off, stream_off, k_max, send, send_capacity, step_off, dev_status, ws, ws_bytes,
                           stream);
}

vp_status vp_pack_prepare_heads(const void* act, int64_t T, int64_t token_stride, const int64_t* head_lo,
                                int64_t head_bytes, int32_t self_rank, int32_t n_ranks, const int32_t* K,
                                const int32_t* dst, const int64_t* bytes, const int64_t* send_off,
                                const int64_t* stream_off, int32_t k_max, int64_t send_capacity,
                                int64_t* step_off, int32_t* dev_status, void* ws, size_t ws_bytes,
                                void* stream) {
  return pack_heads_stages(1, act, T, token_stride, head_lo, head_bytes, self_rank, n_ranks, K, dst, bytes,
                           send_off, stream_off, k_max, nullptr, send_capacity, step_off, dev_status, ws,
                           ws_bytes, stream);
}

vp_status vp_pack_gather(const void* src, int64_t unit_bytes, int64_t T, int32_t k, const int32_t* K,
                         const int64_t* step_off, int32_t k_max, void* send, int64_t send_capacity,
                         int32_t* dev_status, void* ws, size_t ws_bytes, void* stream) {
  if (unit_bytes < 16 || unit_bytes % 16 != 0 || k_max < 1 || send_capacity < 0 || T < 0 || k < 0)
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad gather sizes");
  if ((T > 0 && !src) || !K || !step_off || !dev_status || (send_capacity > 0 && !send))
    return set_error(VP_ERR_INVALID_ARGUMENT, "null pointer");
  if (ws_bytes < vp::pack_workspace(k_max, send_capacity, unit_bytes, T, k) || !ws)
    return set_error(VP_ERR_INVALID_ARGUMENT, "workspace too small");
  vp::PackLaunch a{k > 0 ? 0 : 1, 2, src, T, k, unit_bytes, unit_bytes, nullptr, nullptr, nullptr, nullptr, 0, 1,
                   K, nullptr, nullptr, nullptr, nullptr, k_max, send, send_capacity,
                   const_cast<int64_t*>(step_off), dev_status, ws, ws_bytes};
  return vp::launch_pack(a, stream);
}

int64_t vp_slot_bytes(int64_t row_bytes) { return row_bytes < 1 ? 0 : vp::slot_bytes(row_bytes); }

size_t vp_unpack_workspace(int64_t buffer_rows) {
  if (buffer_rows < 0) return 0;
  return vp::unpack_workspace(buffer_rows);
}

vp_status vp_demand_transpose(const int64_t* demand, int32_t n_ranks, int64_t* demand_t, void* stream) {
  if (!demand || !demand_t || n_ranks < 1 || n_ranks > vp::kMaxRanks || demand == demand_t)
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad transpose arguments");
  return vp::launch_transpose(demand, n_ranks, demand_t, stream);
}

namespace {

// Checks shared by the three receive-side / combine calls.
vp_status check_unpack(int64_t row_bytes, int32_t self_rank, int32_t n_ranks, const int32_t* K, const int32_t* dst,
                       const int64_t* bytes, int32_t k_max, int64_t rows_cap, int64_t map_cap,
                       const int32_t* dev_status, const void* ws, size_t ws_bytes) {
  if (row_bytes < 16 || row_bytes % 16 != 0 || n_ranks < 1 || n_ranks > vp::kMaxRanks || self_rank < 0 ||
      self_rank >= n_ranks || k_max < 1 || rows_cap < 0 || map_cap < 0)
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad unpack sizes (row_bytes must be a multiple of 16)");
  if (rows_cap >= (int64_t(1) << 31) || map_cap >= (int64_t(1) << 31))
    return set_error(VP_ERR_UNSUPPORTED, "more than 2^31 rows");
  if (!K || !dst || !bytes || !dev_status) return set_error(VP_ERR_INVALID_ARGUMENT, "null pointer");
  if (ws_bytes < vp::unpack_workspace(rows_cap) || !ws) return set_error(VP_ERR_INVALID_ARGUMENT, "workspace too small");
  return VP_OK;
}

}  // namespace

vp_status vp_unpack_rows(const void* recv, int64_t recv_capacity, int64_t row_bytes, const int32_t* counts,
                         int32_t E, int32_t self_rank, int32_t n_ranks, const int32_t* K, const int32_t* dst,
                         const int64_t* bytes, const int32_t* recv_src, int32_t k_max, void* out,
                         int64_t out_capacity, int32_t* dev_status, void* ws, size_t ws_bytes, void* stream) {
  const int64_t sb = vp::slot_bytes(row_bytes);
  if (recv_capacity < 0 || out_capacity < 0 || E < 1 || n_ranks < 1 || E % n_ranks != 0 || E > 4096)
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad unpack sizes (E a multiple of N, <= 4096)");
  const int64_t rows_cap = recv_capacity / sb, map_cap = out_capacity / sb;
  vp_status st = check_unpack(row_bytes, self_rank, n_ranks, K, dst, bytes, k_max, rows_cap, map_cap, dev_status,
                              ws, ws_bytes);
  if (st != VP_OK) return st;
  if (!counts || !recv_src || (rows_cap > 0 && (!recv || !out)))
    return set_error(VP_ERR_INVALID_ARGUMENT, "null pointer");
  if (vp::unpack_lds_bytes(vp::kModeDispatchUnpack, n_ranks, E / n_ranks) > 64 * 1024)
    return set_error(VP_ERR_UNSUPPORTED, "too many ranks or local experts for the row map");
  vp::UnpackLaunch a{vp::kModeDispatchUnpack, recv, sb, out, sb, row_bytes, rows_cap, map_cap, self_rank, n_ranks,
                     k_max, E, 0, 0, K, dst, recv_src, bytes, counts, nullptr, nullptr, nullptr, nullptr,
                     dev_status, ws, ws_bytes};
  return vp::launch_unpack(a, stream);
}

vp_status vp_pack_combine(const void* out, int64_t out_capacity, int64_t row_bytes, const int32_t* counts,
                          int32_t E, int32_t self_rank, int32_t n_ranks, const int32_t* K, const int32_t* dst,
                          const int64_t* bytes, int32_t k_max, void* send, int64_t send_capacity,
                          int64_t* step_off, int32_t* dev_status, void* ws, size_t ws_bytes, void* stream) {
  const int64_t sb = vp::slot_bytes(row_bytes);
  if (send_capacity < 0 || out_capacity < 0 || E < 1 || n_ranks < 1 || E % n_ranks != 0 || E > 4096)
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad combine sizes (E a multiple of N, <= 4096)");
  const int64_t rows_cap = send_capacity / row_bytes, map_cap = out_capacity / sb;
  vp_status st = check_unpack(row_bytes, self_rank, n_ranks, K, dst, bytes, k_max, rows_cap, map_cap, dev_status,
                              ws, ws_bytes);
  if (st != VP_OK) return st;
  if (!counts || !step_off || (rows_cap > 0 && (!out || !send)))
    return set_error(VP_ERR_INVALID_ARGUMENT, "null pointer");
  if (vp::unpack_lds_bytes(vp::kModeCombinePack, n_ranks, E / n_ranks) > 64 * 1024)
    return set_error(VP_ERR_UNSUPPORTED, "too many ranks or local experts for the row map");
  vp::UnpackLaunch a{vp::kModeCombinePack, out, sb, send, row_bytes, row_bytes, rows_cap, map_cap, self_rank,
                     n_ranks, k_max, E, 0, 0, K, dst, nullptr, bytes, counts, nullptr, nullptr, nullptr, step_off,
                     dev_status, ws, ws_bytes};
  return vp::launch_unpack(a, stream);
}

vp_status vp_unpack_combine(const void* recv, int64_t recv_capacity, int64_t row_bytes, int64_t T, int32_t k,
                            const int32_t* sorted_tok, const uint8_t* sorted_slot, const int64_t* dest_off,
                            int32_t self_rank, int32_t n_ranks, const int32_t* K, const int32_t* dst,
                            const int64_t* bytes, const int32_t* recv_src, int32_t k_max, void* combined,
                            int32_t* dev_status, void* ws, size_t ws_bytes, void* stream) {
  const int64_t sb = vp::slot_bytes(row_bytes);
  if (recv_capacity < 0 || T < 0 || k < 1 || k > 255)
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad combine sizes (k <= 255)");
  const int64_t rows_cap = recv_capacity / sb, map_cap = T * k;
  vp_status st = check_unpack(row_bytes, self_rank, n_ranks, K, dst, bytes, k_max, rows_cap, map_cap, dev_status,
                              ws, ws_bytes);
  if (st != VP_OK) return st;
  if (!dest_off || !recv_src || (rows_cap > 0 && !recv) || (map_cap > 0 && (!sorted_tok || !sorted_slot || !combined)))
    return set_error(VP_ERR_INVALID_ARGUMENT, "null pointer");
  vp::UnpackLaunch a{vp::kModeCombineUnpack, recv, sb, combined, sb, row_bytes, rows_cap, map_cap, self_rank,
                     n_ranks, k_max, n_ranks, k, T, K, dst, recv_src, bytes, nullptr, sorted_tok, sorted_slot,
                     dest_off, nullptr, dev_status, ws, ws_bytes};
  return vp::launch_unpack(a, stream);
}

vp_status vp_modeled_time(const vp_catalog* c, int32_t K, const int32_t* inst, const int64_t* bytes,
                          int64_t lambda_ns, int64_t* num, int64_t* den) {
  if (!c || K < 0 || (K > 0 && (!inst || !bytes)) || !num || !den || lambda_ns < 0)
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad modeled-time arguments");
  // common denominator of the path rates
  int64_t l = 1;
  for (int64_t bw : c->ibw) {
    int64_t a = l, b = bw;
    while (b) { int64_t t = a % b; a = b; b = t; }
    l = l / a * bw;
  }
  __int128 total = 0;
  for (int k = 0; k < K; ++k) {
    __int128 worst = 0;
    for (int i = 0; i < c->N; ++i) {
      int32_t id = inst[(size_t)k * c->N + i];
      if (id < 0 || id >= (int32_t)c->ibw.size()) return set_error(VP_ERR_INVALID_ARGUMENT, "instance id");
      __int128 v = (__int128)bytes[(size_t)k * c->N + i] * (l / c->ibw[id]);
      worst = std::max(worst, v);
    }
    total += (__int128)lambda_ns * l + worst;
  }
  if (total > (__int128)INT64_MAX) return set_error(VP_ERR_UNSUPPORTED, "modeled time overflows");
  *num = (int64_t)total;
  *den = l;
  return VP_OK;
}

vp_status vp_rotation_time(const vp_catalog* c, const int64_t* demand, int32_t path_rule, int64_t lambda_ns,
                           int64_t* num, int64_t* den) {
  if (!c || !demand || !num || !den || lambda_ns < 0 || (path_rule != 0 && path_rule != 1))
    return set_error(VP_ERR_INVALID_ARGUMENT, "bad rotation-time arguments");
  for (int64_t x = 0; x < (int64_t)c->N * c->N; ++x)
    if (demand[x] < 0) return set_error(VP_ERR_INVALID_ARGUMENT, "negative demand");
  return vp::rotation_time(*c, demand, path_rule, lambda_ns, num, den);
}

}  // extern "C"
