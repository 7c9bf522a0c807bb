// Internal declarations shared by the library's translation units.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>
#include <vector>

#include "../../include/vp.h"

namespace vp {

// Limits of the device planner (checked on the host before any launch).
constexpr int kMaxGpusPerSwitch = 4;
constexpr int kMaxSlotsPerNode = 8;
constexpr int kMaxRanks = 1024;
constexpr int kMaxNodes = 256;
constexpr int kMaxStarts = 16;
constexpr int kPlanThreads = 1024;
constexpr int kMaxRTerms = 8;   // NIC lanes of one node-local pattern (one per source slot)

// Sentinel credit of a self pair (never bindable).
constexpr uint32_t kForbidden = 0xFFFFFFFFu;

// Device image of the catalog: one int32 buffer, sections at these offsets
// (in int32 elements).  A "pattern" is a node-local shape: patterns
// [0, J0) are the intra-node shapes (shift 0), patterns [J0, J0+J1) the
// NIC-carrying shapes repeated for every shift 1..n_nodes-1.  Local
// families [0, F0) belong to shift 0, [F0, F0+F1) to every non-zero shift.
struct DevCatalogLayout {
  int32_t N, G, g, Q, nn, n_inst;
  int32_t J0, J1, F0, F1;
  int32_t TS;            // term slots per pattern
  int32_t n_perm;        // g!
  int64_t J, F;          // global shape / family counts
  int32_t off_terms;     // (J0+J1) * TS packed terms: count | q2<<4 | q<<8 | block<<12
  int32_t off_nterms;    // (J0+J1)
  int32_t off_fb, off_fe;      // (J0+J1) local family range of each pattern
  int32_t off_fam_info;  // (F0+F1) * Q*g : cls | src_slot<<4 | dst_slot<<8 | local_id<<12
  int32_t off_fam_out;   // (F0+F1) * Q*g : [slot][m] local index of the m-th out-instance
  int32_t off_fam_in;    // (F0+F1) * Q*g : [slot][m] local index of the m-th in-instance
  int32_t off_perms;     // n_perm * g, lexicographic order
  int32_t nS;            // distinct NIC-lane sets of the NIC-carrying patterns
  int32_t off_rset;      // nS * kMaxRTerms slot-pair indices q*Q+q2 of each set (-1 past its end)
  int32_t off_psid;      // J1: set of each NIC-carrying pattern
  int32_t total;         // int32 elements
  int64_t bw_cls[4];     // rate of PIX, PXB, NIC, SYS paths
  int64_t bw_max;
};

}  // namespace vp

struct vp_catalog {
  vp_topology topo;
  int N, G, g, Q, nn;
  // node-local instance table (id order)
  std::vector<int32_t> icls, isrc, idst, icopy;
  std::vector<int64_t> ibw;
  // node-local patterns: [0, J0) shift 0, [J0, J0+J1) NIC-carrying
  int J0 = 0, J1 = 0;
  std::vector<std::vector<int32_t>> patL, patR;
  std::vector<int32_t> pat_fb, pat_fe;
  // node-local families: [0, F0) shift 0, [F0, F0+F1) NIC-carrying
  int F0 = 0, F1 = 0;
  std::vector<std::vector<int32_t>> lfam;
  // device copy
  vp::DevCatalogLayout lay{};
  std::vector<int32_t> image;
  void* dev = nullptr;
  int dev_id = -1;
};

namespace vp {

vp_status set_error(vp_status s, const std::string& msg);
vp_status build_catalog_host(const vp_topology& t, vp_catalog& c);
std::vector<uint8_t> serialize_catalog(const vp_catalog& c);
vp_status restrict_catalog(const vp_catalog& in, int rule, vp_catalog& out);
vp_status rotation_time(const vp_catalog& c, const int64_t* D, int rule, int64_t lambda, int64_t* num,
                        int64_t* den);
vp_status deserialize_catalog(const uint8_t* p, size_t n, vp_catalog& c,
                              vp_status (*check_topology)(const vp_topology&));
void build_device_image(vp_catalog& c);

struct PlanLaunch {
  const vp_catalog* cat;
  const int64_t* demand;
  int64_t* drem;
  vp_plan_params p;
  int32_t *K, *family, *dst, *inst;
  int64_t *bytes, *tau;
  int64_t *send_off, *stream_off;
  int32_t* recv_src;
  int32_t* status;
  int32_t batch;   // matrices planned side by side, one workgroup each
};
vp_status launch_plan(const PlanLaunch& a, void* stream);
// Ranks the library-owned residual of vp_plan_noalloc holds, and its device
// address on the current device (looked up on the first call per device).
constexpr int kStaticRanks = 256;
vp_status static_residual(int32_t n_ranks, void** out);

struct DemandLaunch {
  const int32_t* routing;
  int32_t R;
  int64_t T;
  int32_t k, E, N, first_rank, sort_row;
  int64_t unit;
  int32_t* counts;
  int64_t* demand;
  int32_t* sorted_tok;
  uint8_t* sorted_slot;
  int64_t* dest_off;
  int32_t* status;
  void* ws;
  size_t ws_bytes;
};
size_t demand_workspace(int32_t R, int64_t T, int32_t k, int32_t E);
vp_status launch_demand(const DemandLaunch& a, void* stream);
vp_status launch_control_words(const int32_t* counts, int32_t R, int32_t E, int32_t N, int32_t first_rank,
                               uint32_t* words, int32_t* status, void* stream);
vp_status launch_receive_counts(const uint32_t* words, int64_t word_stride, const int32_t* signal, int32_t N,
                                int32_t L, int32_t* counts, void* stream);
vp_status launch_demand_heads(int64_t T, const int64_t* head_lo, int64_t head_bytes, int32_t N,
                              int32_t first_rank, int32_t R, int64_t* demand, int32_t* status,
                              void* stream);

struct PackLaunch {
  int mode;    // 0 rows, 1 heads
  int stages;  // 1 prepare (slice + index kernels), 2 gather, 3 both
  const void* src;
  int64_t T;
  int32_t k;   // rows: routing top-k (copies per token at most); heads: 0
  int64_t unit, token_stride;
  const int32_t* sorted_tok;
  const uint8_t* sorted_slot;
  const int64_t* dest_off;
  const int64_t* head_lo;
  int32_t self_rank, N;
  const int32_t *K, *dst;
  const int64_t* bytes;
  const int64_t *send_off, *stream_off;   // the planner's buffer layout, or both null
  int32_t k_max;
  void* send;
  int64_t send_capacity;
  int64_t* step_off;
  int32_t* status;
  void* ws;
  size_t ws_bytes;
};
size_t pack_workspace(int32_t k_max, int64_t send_capacity, int64_t unit, int64_t T, int32_t k);
vp_status launch_pack(const PackLaunch& a, void* stream);

// Receive side and combine direction.  The buffer side holds rows in step
// order (receive slots, or the combine's send rows); the mapped side is the
// expert-major output or the [T, k] combine output.
enum { kModeDispatchUnpack = 0, kModeCombinePack = 1, kModeCombineUnpack = 2 };
struct UnpackLaunch {
  int mode;
  const void* src;
  int64_t src_stride;
  void* dst_buf;
  int64_t dst_stride;
  int64_t row_bytes;
  int64_t rows_cap, map_cap;
  int32_t self_rank, N, k_max, E, k;
  int64_t T;
  const int32_t *K, *dst, *recv_src;
  const int64_t* bytes;
  const int32_t* counts;
  const int32_t* sorted_tok;
  const uint8_t* sorted_slot;
  const int64_t* dest_off;
  int64_t* step_off;
  int32_t* status;
  void* ws;
  size_t ws_bytes;
};
int64_t slot_bytes(int64_t row_bytes);
size_t unpack_workspace(int64_t rows);
size_t unpack_lds_bytes(int mode, int32_t N, int32_t eloc);
vp_status launch_unpack(const UnpackLaunch& a, void* stream);
vp_status launch_transpose(const int64_t* D, int32_t N, int64_t* DT, void* stream);

}  // namespace vp
