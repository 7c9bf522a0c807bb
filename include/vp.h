/* vp.h -- C-ABI of the VarioPath demand -> plan -> pack hot path for MI355X.
 *
 * The library turns one AlltoAllv invocation's routing into
 *   (1) an N x N byte-demand matrix            (Sec. 3 "Model setup"),
 *   (2) an ordered list of channel activations  (Sec. 4.2, Alg. 2),
 *   (3) channel-ordered send buffers            (Sec. 5 "Device-resident buffer layout"),
 * against an offline catalog of contention-free channel families
 * (Sec. 4.1, Alg. 1), and unpacks received buffers into the output layout,
 * for the dispatch and for the combine that returns the rows.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Pointers marked "device" are HIP device allocations owned by the caller
 *   (e.g. torch tensors passed by data_ptr()).  Pointers marked "host" are
 *   ordinary host memory owned by the caller.  The library owns only the
 *   opaque vp_catalog handle, released with vp_catalog_free().
 * - `stream` is a hipStream_t passed as void*; NULL means the default stream.
 *   Every device entry point only enqueues work on that stream and returns
 *   without synchronising.  No hot call allocates memory: scratch space comes
 *   from the caller through a workspace pointer whose size is given by the
 *   matching *_workspace() query.
 * - Errors found on the host (bad sizes, null pointers, unsupported shapes)
 *   are returned immediately and nothing is enqueued.  Errors that only the
 *   device can see (an expert id out of range, a demand entry that is
 *   negative, on the diagonal or not a multiple of the unit, a plan that
 *   cannot progress or exceeds k_max, a pack slice outside its stream) are
 *   written to the caller's device int32 `dev_status` (first error wins,
 *   VP_OK = 0 means none) and become visible after the stream is
 *   synchronised.  Kernels never trap; after a device error the outputs of
 *   that call are unspecified.  The caller clears dev_status (write 0)
 *   before a chain of calls.  Nothing throws or aborts across this ABI.
 * - vp_last_error() returns a thread-local text for the last host-side
 *   error of the calling thread.
 */
#ifndef VP_H_
#define VP_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  VP_OK = 0,
  VP_ERR_INVALID_ARGUMENT = 1, /* bad pointer/size, or a routing id outside [0, E) */
  VP_ERR_INVALID_DEMAND = 2,   /* D_ij < 0, D_ii != 0, or D_ij not a multiple of the unit */
  VP_ERR_NO_PROGRESS = 3,      /* an iteration of Alg. 2 could serve no byte */
  VP_ERR_CAPACITY = 4,         /* schedule longer than k_max, or send buffer too small */
  VP_ERR_UNSUPPORTED = 5,      /* shape outside the library's limits (see each call) */
  VP_ERR_HIP = 6               /* a HIP runtime call failed */
} vp_status;

/* Path classes of a lane (Sec. 3; Fig. 1 legend): same switch, same socket
 * through the root complex, through the switches' NICs, and (with
 * VP_TOPO_SYS_P2P) between sockets of one node through both root complexes
 * and the inter-socket link. */
enum { VP_PATH_PIX = 0, VP_PATH_PXB = 1, VP_PATH_NIC = 2, VP_PATH_SYS = 3 };

/* vp_topology.flags.  VP_TOPO_SYS_P2P: GPUs under different sockets of one
 * node reach each other peer to peer (path class SYS: the source switch's
 * uplink, the directed link from the source socket to the destination
 * socket, the destination switch's downlink; PCIe rate).  Without it such
 * pairs go through the NICs only. */
enum { VP_TOPO_SYS_P2P = 1 };

/* A PCIe cluster (Sec. 3 "Model setup", Sec. 5 "Topology, path, and rate
 * model").  Rank = ((node * sockets + socket) * switches + switch) * gpus + local;
 * one rank group per PCIe switch.  Each switch has nics_per_switch NICs, all
 * reachable from every GPU of the switch: a NIC path leaves through one NIC
 * of the source switch (its transmit side) and arrives through one NIC of
 * the destination switch (its receive side).  Families that differ only by
 * which of a switch's NICs their lanes use are one family (the catalog
 * keeps the one with the smallest instance ids).  Rates are in bytes per
 * nanosecond; a NIC path runs at min(pcie, nic), PIX, PXB and SYS paths at
 * the PCIe rate.
 * Limits of the library: gpus_per_switch in [2, 4], sockets*switches <= 8,
 * nics_per_switch in [1, 4] with 2*Q*(1 + nics) (+ sockets^2 with SYS) <= 64
 * for Q = sockets*switches, at most 256 node-local path instances, n_nodes
 * in [1, 256], N <= 1024.  vp_rotation_time takes one NIC per switch. */
typedef struct {
  int32_t n_nodes;
  int32_t sockets_per_node;
  int32_t switches_per_socket;
  int32_t gpus_per_switch;
  int32_t nics_per_switch;
  int32_t flags;               /* 0 or VP_TOPO_SYS_P2P (then sockets_per_node <= 4) */
  int64_t pcie_bytes_per_ns;
  int64_t nic_bytes_per_ns;
} vp_topology;

/* Inputs of Alg. 2 (Sec. 4.2) and of the quantum of Sec. 5 "Global execution
 * granularity".  vp_plan_params_default() fills K_target = 2N, lambda =
 * 10,000 ns, N_start = 4, I_AA = 8, seed = 0, k_max = 8N. */
typedef struct {
  int64_t k_target;    /* target round count; tau = ceil(L_max / (bw_max * k_target)) ns */
  int64_t lambda_ns;   /* fixed per-activation overhead of Eq. (2) and Eq. (10) */
  int64_t unit_bytes;  /* pack granule; every demand entry is a multiple of it */
  int32_t n_start;     /* MultiStartAA starts, 1..16 */
  int32_t i_aa;        /* AA sweep limit, >= 0 */
  uint64_t seed;       /* key of the counter-based random starts */
  int32_t k_max;       /* capacity of the schedule arrays (rows) */
  int32_t reserved;
} vp_plan_params;

typedef struct vp_catalog vp_catalog; /* opaque, library-owned */

/* ---------------------------------------------------------------- catalog */

/* Offline catalog construction (Sec. 4.1, Alg. 1, PrunePaths, PruneFamilies),
 * host only.  For one node this is the full Alg. 1 catalog; for several nodes
 * it is the node-circulant catalog: a family repeats one node-local pattern in
 * every node with all NIC lanes of node n landing on node (n + k) mod n_nodes.
 * Shapes are ordered by (k, diagonal node block, shift node block) and
 * families inside a shape by their sorted node-local instance ids.
 * *out receives a new handle (free with vp_catalog_free).  A node whose
 * candidate channel sets exceed 2^22 before pruning (one node of eight
 * switches of two GPUs already does) returns VP_ERR_UNSUPPORTED after a few
 * seconds instead of exhausting host memory. */
vp_status vp_build_catalog(const vp_topology* topo, vp_catalog** out);

/* info[0..7] = N, G (groups), g, Q (switches per node), n_nodes, shapes,
 * families, node-local instances.  Host only. */
vp_status vp_catalog_info(const vp_catalog* cat, int64_t info[8]);

/* Node-local instance table in id order (host arrays of length info[7]):
 * path class, source slot, destination slot, copy index, rate (bytes/ns). */
vp_status vp_catalog_instances(const vp_catalog* cat, int32_t* cls, int32_t* src_slot,
                               int32_t* dst_slot, int32_t* copy, int64_t* bw);

/* Canonical shapes (host arrays, J = info[5], Q = info[3]): node shift k,
 * family range [fam_begin, fam_end), and the Q x Q lane counts of the
 * diagonal node block (L) and of the block from node n to node n+k (R). */
vp_status vp_catalog_shapes(const vp_catalog* cat, int32_t* k, int32_t* fam_begin,
                            int32_t* fam_end, int32_t* L, int32_t* R);

/* Canonical families (host arrays, F = info[6]): shape index, node shift k,
 * and the Q*g node-local instance ids of each family, ascending. */
vp_status vp_catalog_families(const vp_catalog* cat, int32_t* shape, int32_t* k, int32_t* ids);

/* Restricted catalogs for the peer/path ablation (Sec. 6.3, Table 3): a new
 * handle holding the families of `cat` that satisfy `rule`, in the same
 * canonical order.  VP_RESTRICT_NEAREST_PATH keeps the families in which
 * every lane takes its group pair's nearest path (PIX inside a switch, PXB
 * between two switches of one socket, SYS between sockets when enabled, the
 * NICs otherwise), i.e. drops every family with a NIC lane between two
 * switches of one node that a PCIe peer-to-peer path also joins ("fixed
 * nearest path, demand-aware peers").  Host only; free with vp_catalog_free.  An
 * unknown rule returns VP_ERR_INVALID_ARGUMENT. */
enum { VP_RESTRICT_NEAREST_PATH = 1 };
vp_status vp_catalog_restrict(const vp_catalog* cat, int32_t rule, vp_catalog** out);

/* Compact serialized catalog (Table 4 sizes the catalog tree by such a
 * payload): the topology and the node-local instance ids of every family,
 * little-endian, with a 64-bit FNV-1a hash at the end; see vp_catalog_load.
 * With buf == NULL, *size receives the byte count and nothing else happens;
 * otherwise `buf` (host, `capacity` bytes, caller-owned) receives the payload
 * and *size its length, or VP_ERR_CAPACITY when capacity is too small.  Host
 * only. */
vp_status vp_catalog_save(const vp_catalog* cat, void* buf, size_t capacity, size_t* size);

/* A new catalog handle from a payload written by vp_catalog_save (host
 * memory, `size` bytes), without running Alg. 1 again.  Everything Alg. 1
 * guarantees is checked: the hash, the topology limits, and for every family
 * that it is a complete (g lanes out of and into every switch slot),
 * resource-disjoint set of instances that PrunePaths keeps (Eq. (1),
 * Eq. (4)), identical PIX copies in copy order, a NIC lane in every
 * shifted-node family, and strictly increasing canonical order.  A subset of
 * the families Alg. 1 finds is accepted (a restricted catalog; the planner
 * then reports VP_ERR_NO_PROGRESS for demand no family can serve).  Any
 * failure returns VP_ERR_INVALID_ARGUMENT (VP_ERR_UNSUPPORTED for topology
 * limits) and leaves *out NULL.  Free the handle with vp_catalog_free. */
vp_status vp_catalog_load(const void* buf, size_t size, vp_catalog** out);

/* Copy the catalog to the current device once (synchronous on `stream`);
 * the device copy belongs to the handle.  Needed before vp_plan. */
vp_status vp_catalog_upload(vp_catalog* cat, void* stream);

void vp_catalog_free(vp_catalog* cat);

/* ----------------------------------------------------------------- demand */

/* Workspace bytes for vp_demand over `R` rows of `T` tokens, top-`k`, `E`
 * experts: the partial expert counts of each part of each row and the
 * sorted row's chunk counts.  It needs no clearing; calls that share a
 * workspace must not overlap.  Returns 0 for bad sizes. */
size_t vp_demand_workspace(int32_t R, int64_t T, int32_t k, int32_t E);

/* Demand rows from routing (Sec. 3 model setup; one row copy per (token,
 * expert) assignment, Sec. 5 sparse EP).  For R source ranks
 * first_rank .. first_rank+R-1:
 *   routing    device int32 [R, T, k]  expert ids in [0, E)
 *   counts     device int32 [R, E]     assignments per expert
 *   demand     device int64 [R, N]     D_r,j = unit * sum of counts of the
 *                                      E/N experts hosted by rank j
 *                                      (experts contiguous per rank),
 *                                      D_r,r = 0
 * and for row `sort_row` (0 <= sort_row < R, or -1 for none):
 *   sorted_tok device int32 [T*k]      token ids of that row's assignments in
 *                                      (expert, token) order (stable)
 *   sorted_slot device uint8 [T*k]     the routing slot (0..k-1) of each of
 *                                      those assignments; may be NULL
 *   dest_off   device int64 [N+1]      first position of each destination
 *                                      rank's rows in sorted_tok
 * E must be a positive multiple of N, E <= 4096, k <= 255, T*k < 2^31.  An
 * expert id outside [0, E) sets VP_ERR_INVALID_ARGUMENT in dev_status. */
vp_status vp_demand(const int32_t* routing, int32_t R, int64_t T, int32_t k, int32_t E,
                    int32_t n_ranks, int32_t first_rank, int32_t sort_row, int64_t unit_bytes,
                    int32_t* counts, int64_t* demand, int32_t* sorted_tok, uint8_t* sorted_slot,
                    int64_t* dest_off, int32_t* dev_status, void* ws, size_t ws_bytes, void* stream);

/* Ulysses head/context re-layout demand (Sec. 6.2 sequence parallelism):
 * rank j owns heads [head_lo[j], head_lo[j+1]) (device int64 [N+1]); each of
 * the T local tokens sends its heads of rank j there:
 *   demand device int64 [R, N], D_r,j = T * (head_lo[j+1]-head_lo[j]) * head_bytes,
 *   D_r,r = 0, for ranks first_rank .. first_rank+R-1.
 * A decreasing head_lo sets VP_ERR_INVALID_ARGUMENT in dev_status. */
vp_status vp_demand_heads(int64_t T, const int64_t* head_lo, int64_t head_bytes, int32_t n_ranks,
                          int32_t first_rank, int32_t R, int64_t* demand, int32_t* dev_status,
                          void* stream);

/* Sparse expert-parallel control words (Sec. 5 "Efficient sparse data
 * movement for expert parallelism").  Rank j hosts L = E/N local experts
 * (experts j*L .. j*L+L-1).  For each of R source ranks
 * first_rank .. first_rank+R-1 and every destination j:
 *   counts device int32 [R, E]    per-expert row counts (as vp_demand writes)
 *   words  device uint32 [R, N]   bit l (l < L) set when the source sends at
 *                                 least one row to local expert l of rank j;
 *                                 bits L..31 hold the exact row count of the
 *                                 designated expert, the highest active one
 *                                 (its payload ends the pair's expert-
 *                                 ascending stream, the word follows it).
 *                                 0 for the self pair and for pairs with no
 *                                 rows: no transfer and no wait.
 * L <= 31, else VP_ERR_UNSUPPORTED.  A designated count that does not fit in
 * 32 - L bits sets VP_ERR_CAPACITY, a negative count VP_ERR_INVALID_ARGUMENT,
 * in dev_status (that pair's word is then 0). */
vp_status vp_control_words(const int32_t* counts, int32_t R, int32_t E, int32_t n_ranks, int32_t first_rank,
                           uint32_t* words, int32_t* dev_status, void* stream);

/* The receiver's decode of the same words (Sec. 5): rank r holds the word of
 * every source i at words[i * word_stride] (device uint32; word_stride = 1
 * for a gathered vector, N for column r of vp_control_words' output) and the
 * per-expert signal counts signal[i][l] (device int32 [N, L]), which are read
 * only for active experts other than the designated one.  Writes
 *   counts device int32 [N, L]: rows from source i for local expert l
 *   (0 where the bitmap bit is clear, the word's count for the designated
 *   expert, the signal's otherwise).
 * 1 <= n_local <= 31. */
vp_status vp_receive_counts(const uint32_t* words, int64_t word_stride, const int32_t* signal, int32_t n_ranks,
                            int32_t n_local, int32_t* counts, void* stream);

/* ------------------------------------------------------------------- plan */

void vp_plan_params_default(int32_t n_ranks, int64_t unit_bytes, vp_plan_params* p);

/* Workspace bytes for vp_plan (holds the residual demand D^rem). */
size_t vp_plan_workspace(const vp_catalog* cat, const vp_plan_params* p);

/* Online channel-guided demand decomposition (Sec. 4.2, Alg. 2), run
 * entirely on the device by one persistent kernel:
 *   demand  device int64 [N, N]  bytes from rank i (row) to rank j (column)
 *   K       device int32 [1]     activations emitted
 *   family  device int32 [k_max] global family index of each activation
 *   dst     device int32 [k_max, N]  pi_k(i) for source rank i
 *   inst    device int32 [k_max, N]  node-local instance id of lane i
 *   bytes   device int64 [k_max, N]  x_{k,i} of Eq. (9) (zero lanes kept)
 *   send_off, stream_off  device int64 [k_max, N], both NULL or both given:
 *           the buffer layout of Sec. 5 for every rank i: bytes i sent in the
 *           steps before k (where step k's slice starts in i's send buffer),
 *           and bytes i sent to pi_k(i) before step k (where the slice starts
 *           in i's stream to that destination)
 *   recv_src device int32 [k_max, N], may be NULL: the receive view of the
 *           same steps, recv_src[k, j] = the rank i with pi_k(i) = j (every
 *           step is a permutation, so each entry below K is written once);
 *           the unpack calls below take it
 *   tau     device int64 [1]     the quantum used (ns), may be NULL
 * Each iteration scores every catalog shape (Eq. (5)-(6)), binds every family
 * of the best shape with MultiStartAA (Eq. (7)-(8)), evaluates Eq. (9)-(10)
 * exactly and appends the best activation.  Device errors:
 * VP_ERR_INVALID_DEMAND, VP_ERR_NO_PROGRESS, VP_ERR_CAPACITY, and
 * VP_ERR_UNSUPPORTED when a demand entry reaches 2^42 bytes, a capacity
 * tau*bw reaches 2^31 bytes or 2^27 units, or the total demand reaches 2^42
 * bytes or 2^28 units (the planner keeps unit counts in 32 bits: 4 GiB of
 * demand at a 16-byte unit, 64 GiB at a 256-byte unit).  An invalid entry
 * takes precedence over these limits.  The catalog must have been uploaded.  Host
 * errors, returned before anything is enqueued: VP_ERR_UNSUPPORTED when
 * k_max * N * 8 reaches 2^32 (one matrix's schedule arrays are addressed with
 * 32-bit byte offsets), when the catalog exceeds the kernel's index widths
 * (more than 4095 shapes of either kind, 255 node shifts, 256 node-local
 * instances, 512 rank groups, 8 switches per node or 4 GPUs per switch, or a
 * pattern with more intra-node lane classes or NIC lanes than its term
 * tables hold), and when the planner's
 * per-catalog state (shape terms, family lane maps, node aggregates) plus one
 * family's working set does not fit in one workgroup's LDS (160 KiB on gfx950):
 * two-socket nodes of two switches of three GPUs with cross-socket peer to
 * peer (2,744 families over 2,185 shapes from two nodes on) are the smallest
 * such catalogs met.  Larger catalogs need a planner that keeps those tables
 * in HBM. */
vp_status vp_plan(const vp_catalog* cat, const int64_t* demand, const vp_plan_params* p,
                  int32_t* K, int32_t* family, int32_t* dst, int32_t* inst, int64_t* bytes,
                  int64_t* send_off, int64_t* stream_off, int32_t* recv_src, int64_t* tau,
                  int32_t* dev_status, void* ws, size_t ws_bytes, void* stream);

/* vp_plan without a workspace, for callers that cannot allocate device
 * memory around the call (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation): the same arguments, decisions
 * and outputs as vp_plan, with the residual D^rem kept in a device array
 * that the library owns (8 * 256 * 256 bytes, one copy per device, held
 * until the process ends).  The first call on a device looks the array up
 * (do it once outside any capture); no call allocates.  Catalogs of more
 * than 256 ranks return VP_ERR_UNSUPPORTED before anything is enqueued.
 * Every call on a device shares the one array: calls that overlap on one
 * device (other streams, other threads) race and must be serialised by the
 * caller.  Nothing in the array needs clearing (the residual is rewritten
 * from the demand at the start of every call). */
vp_status vp_plan_noalloc(const vp_catalog* cat, const int64_t* demand, const vp_plan_params* p,
                          int32_t* K, int32_t* family, int32_t* dst, int32_t* inst, int64_t* bytes,
                          int64_t* send_off, int64_t* stream_off, int32_t* recv_src, int64_t* tau,
                          int32_t* dev_status, void* stream);

/* Several independent matrices planned side by side, one workgroup (one
 * compute unit) each, with the decisions vp_plan takes for each of them (the
 * planner is latency-bound on one CU; a batch puts the others to work, e.g.
 * a layer's dispatch matrix D and its combine matrix D^T, or a stream of
 * matrices planned ahead).  Every buffer of vp_plan holds `batch` of its
 * kind back to back: demand [batch, N, N]; K, tau and dev_status [batch];
 * family [batch, k_max]; dst, inst, bytes and the optional send_off,
 * stream_off, recv_src [batch, k_max, N].  Matrix b's device errors land in
 * dev_status[b].  Workspace: vp_plan_batch_workspace bytes (batch * N * N *
 * 8).  1 <= batch <= 65535. */
size_t vp_plan_batch_workspace(const vp_catalog* cat, const vp_plan_params* p, int32_t batch);
vp_status vp_plan_batch(const vp_catalog* cat, int32_t batch, const int64_t* demand, const vp_plan_params* p,
                        int32_t* K, int32_t* family, int32_t* dst, int32_t* inst, int64_t* bytes,
                        int64_t* send_off, int64_t* stream_off, int32_t* recv_src, int64_t* tau,
                        int32_t* dev_status, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------------------------- pack */

/* Workspace bytes for vp_pack_rows (k = the routing's top-k, T tokens) or
 * vp_pack_heads (k = 0) with schedule capacity k_max, a send buffer of
 * send_capacity bytes and a pack unit of unit_bytes (row_bytes or
 * head_bytes).  Rows: per-step descriptors and one send-unit entry per
 * (token, routing slot).  Heads: per-step descriptors only.  The workspace
 * must be zero-filled once before its first use; no later call needs it
 * cleared (rows: the entries carry the generation of the call that wrote
 * them).  Returns 0 for negative sizes. */
size_t vp_pack_workspace(int32_t k_max, int64_t send_capacity, int64_t unit_bytes, int64_t T, int32_t k);

/* Send-buffer layout (Sec. 5 "Device-resident buffer layout"): for the steps
 * in which rank `self_rank` carries bytes, in schedule order, append the next
 * x bytes of the stream to that step's destination.  Stream j is rank
 * self_rank's token rows for j in (expert, token) order:
 *   tokens     device [T, row_bytes]   token rows (bf16 or any bytes)
 *   k                                  top-k of the routing (a token may
 *                                      have at most k copies)
 *   sorted_tok, sorted_slot            from vp_demand ([T*k] each)
 *   dest_off   device int64 [N+1]      from vp_demand (row units)
 *   K, dst, bytes                      the schedule of vp_plan (device)
 *   send_off, stream_off               vp_plan's buffer layout (device), or
 *                                      both NULL: then a slice kernel derives
 *                                      the same offsets from the schedule.
 *                                      The layout must be this schedule's:
 *                                      each step's send offset equal to the
 *                                      previous step's plus its bytes (0 for
 *                                      step 0), else VP_ERR_INVALID_ARGUMENT
 *   send       device [send_capacity]  output
 *   step_off   device int64 [k_max+1]  where step k's slice starts in send;
 *                                      entries past K are unspecified,
 *                                      step_off[K] = total bytes
 * row_bytes must be a multiple of 16 and send_capacity / row_bytes below
 * 2^31; without the planner's layout, k_max is bounded by the slice
 * kernel's LDS table (VP_ERR_UNSUPPORTED).  Each token row is read from HBM
 * once and stored to all its copies.  Slices that are not whole rows or run
 * past their stream, a token id or slot out of range, or a total above
 * send_capacity set VP_ERR_INVALID_ARGUMENT or VP_ERR_CAPACITY in dev_status
 * and write nothing to send.  Calls that share a workspace must not
 * overlap. */
vp_status vp_pack_rows(const void* tokens, int64_t T, int32_t k, int64_t row_bytes, const int32_t* sorted_tok,
                       const uint8_t* sorted_slot, const int64_t* dest_off, int32_t self_rank, int32_t n_ranks,
                       const int32_t* K, const int32_t* dst, const int64_t* bytes, const int64_t* send_off,
                       const int64_t* stream_off, int32_t k_max, void* send, int64_t send_capacity,
                       int64_t* step_off, int32_t* dev_status, void* ws, size_t ws_bytes, void* stream);

/* Ulysses variant: stream j is, token by token, the bytes of the heads rank j
 * owns, [head_lo[j], head_lo[j+1]) (device int64 [N+1]); units are single
 * heads of head_bytes (a multiple of 16); activations are [T, token_stride].
 * Every head a destination owns must lie inside the token row, else
 * VP_ERR_INVALID_ARGUMENT.  With the planner's layout, k_max <= 512 and
 * n_ranks <= 1024 the checks and the copy run as one kernel, in which every
 * workgroup checks the whole schedule before it copies (so an error still
 * writes nothing to send); otherwise the two halves below run.  Limits
 * (VP_ERR_UNSUPPORTED): token_stride / head_bytes at most 2^15, head_bytes
 * below 2^23, token_stride below 2^32, send_capacity below 2^52, and
 * T * (token_stride / head_bytes)^2 and (send_capacity / 16) * (head_bytes /
 * 16) below 2^63. */
vp_status vp_pack_heads(const void* act, int64_t T, int64_t token_stride, const int64_t* head_lo,
                        int64_t head_bytes, int32_t self_rank, int32_t n_ranks, const int32_t* K,
                        const int32_t* dst, const int64_t* bytes, const int64_t* send_off,
                        const int64_t* stream_off, int32_t k_max, void* send, int64_t send_capacity,
                        int64_t* step_off, int32_t* dev_status, void* ws, size_t ws_bytes, void* stream);

/* The two halves of vp_pack_rows / vp_pack_heads, for callers that schedule
 * or time the copy on its own.  vp_pack_prepare_* take the same arguments
 * minus `send` and run the slice (without the planner's layout) and index
 * kernels: they fill step_off and the workspace (the copy lists of every
 * token, or one descriptor per step for heads) and check every slice and
 * the capacity.  vp_pack_gather then copies the units from `src` (the tokens or
 * activations given to the prepare call) into `send` with 16-byte loads and
 * non-temporal stores; it must get the same unit_bytes, T, k (0 after
 * vp_pack_prepare_heads), k_max, send_capacity and workspace, and no other
 * prepare on that workspace may come between.  It writes nothing when
 * dev_status already holds an error.  Heads: every step's descriptor is
 * checked against the activations and the send buffer again before its
 * units are copied, and every unit's source address follows from it. */
vp_status vp_pack_prepare_rows(const void* tokens, int64_t T, int32_t k, int64_t row_bytes,
                               const int32_t* sorted_tok, const uint8_t* sorted_slot,
                               const int64_t* dest_off, int32_t self_rank, int32_t n_ranks,
                               const int32_t* K, const int32_t* dst, const int64_t* bytes,
                               const int64_t* send_off, const int64_t* stream_off, int32_t k_max,
                               int64_t send_capacity, int64_t* step_off, int32_t* dev_status, void* ws,
                               size_t ws_bytes, void* stream);
vp_status vp_pack_prepare_heads(const void* act, int64_t T, int64_t token_stride, const int64_t* head_lo,
                                int64_t head_bytes, int32_t self_rank, int32_t n_ranks, const int32_t* K,
                                const int32_t* dst, const int64_t* bytes, const int64_t* send_off,
                                const int64_t* stream_off, int32_t k_max, int64_t send_capacity,
                                int64_t* step_off, int32_t* dev_status, void* ws, size_t ws_bytes,
                                void* stream);
vp_status vp_pack_gather(const void* src, int64_t unit_bytes, int64_t T, int32_t k, const int32_t* K,
                         const int64_t* step_off, int32_t k_max, void* send, int64_t send_capacity,
                         int32_t* dev_status, void* ws, size_t ws_bytes, void* stream);

/* ------------------------------------------------ receive side, combine */

/* Receive slots (Sec. 5 low-latency protocol): every received row starts at a
 * 128-byte-aligned address; the slot stride is row_bytes rounded up to 128.
 * Returns 0 for row_bytes < 1. */
int64_t vp_slot_bytes(int64_t row_bytes);

/* Workspace bytes of vp_unpack_rows, vp_pack_combine and vp_unpack_combine
 * for a buffer side of `buffer_rows` rows (receive slots, or the combine's
 * send rows): one int32 row index per row and a small header.  It needs no
 * clearing.  Returns 0 for a negative count. */
size_t vp_unpack_workspace(int64_t buffer_rows);

/* D^T (device int64 [N, N], not in place): the demand of the return AlltoAllv
 * of expert parallelism, whose schedule vp_plan computes like any other. */
vp_status vp_demand_transpose(const int64_t* demand, int32_t n_ranks, int64_t* demand_t, void* stream);

/* Dispatch receive (Sec. 5 "Device-resident buffer layout": the receive
 * kernel unpacks straight into the output layout).  Rank self_rank's receive
 * buffer holds the slices addressed to it, in step order, one row per slot of
 * vp_slot_bytes(row_bytes); this call writes every row to the expert-major
 * output:
 *   recv     device [recv_capacity]    received rows
 *   counts   device int32 [N, E]       assignments per (source rank, expert),
 *                                      as vp_demand returns them for R = N
 *   K, dst, bytes                      the dispatch schedule (device)
 *   recv_src device int32 [k_max, N]   vp_plan's receive view of it
 *   out      device [out_capacity]     expert-major output, one row per slot:
 *                                      local expert m (expert self_rank*E/N+m)
 *                                      takes the rows of source 0, then source
 *                                      1, ..., each in token order; the slots
 *                                      of this rank's own rows (never sent)
 *                                      are left untouched
 * row_bytes must be a multiple of 16; the schedule must deliver every source's
 * stream to this rank whole (the rows of its assignments to this rank's
 * experts), else VP_ERR_INVALID_ARGUMENT.  A receive buffer or output too
 * small sets VP_ERR_CAPACITY.  On a device error nothing is copied.  Calls
 * that share a workspace must not overlap. */
vp_status vp_unpack_rows(const void* recv, int64_t recv_capacity, int64_t row_bytes, const int32_t* counts,
                         int32_t E, int32_t self_rank, int32_t n_ranks, const int32_t* K, const int32_t* dst,
                         const int64_t* bytes, const int32_t* recv_src, int32_t k_max, void* out,
                         int64_t out_capacity, int32_t* dev_status, void* ws, size_t ws_bytes, void* stream);

/* Combine send: rank self_rank returns the rows in its expert-major output
 * (layout of vp_unpack_rows, same counts) to their source ranks.  Stream
 * self_rank -> i is source i's rows in (expert, token) order; K, dst, bytes
 * are a schedule planned on the transposed demand.  Slices are appended in
 * step order as by vp_pack_rows:
 *   send     device [send_capacity]    output, rows packed at row_bytes
 *   step_off device int64 [k_max+1]    where step k's slice starts in send;
 *                                      step_off[K] = total bytes
 * Errors as for vp_unpack_rows (every stream must be covered whole). */
vp_status vp_pack_combine(const void* out, int64_t out_capacity, int64_t row_bytes, const int32_t* counts,
                          int32_t E, int32_t self_rank, int32_t n_ranks, const int32_t* K, const int32_t* dst,
                          const int64_t* bytes, int32_t k_max, void* send, int64_t send_capacity,
                          int64_t* step_off, int32_t* dev_status, void* ws, size_t ws_bytes, void* stream);

/* Combine receive at source rank self_rank: the stream from rank r carries
 * the rows of this rank's assignments to r's experts, in the (expert, token)
 * order of its dispatch (sorted_tok, sorted_slot, dest_off from vp_demand);
 * every received row goes to slot (token * k + routing slot) of
 *   combined device [T * k, vp_slot_bytes(row_bytes)]
 * Slots of assignments to this rank's own experts are left untouched.
 * K, dst, bytes, recv_src: the combine schedule and its receive view. */
vp_status vp_unpack_combine(const void* recv, int64_t recv_capacity, int64_t row_bytes, int64_t T, int32_t k,
                            const int32_t* sorted_tok, const uint8_t* sorted_slot, const int64_t* dest_off,
                            int32_t self_rank, int32_t n_ranks, const int32_t* K, const int32_t* dst,
                            const int64_t* bytes, const int32_t* recv_src, int32_t k_max, void* combined,
                            int32_t* dev_status, void* ws, size_t ws_bytes, void* stream);

/* --------------------------------------------------------------- helpers */

/* Modeled completion time of a schedule, Eq. (2), as the exact fraction
 * num/den nanoseconds (host arrays inst, bytes of shape [K, N]). */
vp_status vp_modeled_time(const vp_catalog* cat, int32_t K, const int32_t* inst,
                          const int64_t* bytes, int64_t lambda_ns, int64_t* num, int64_t* den);

/* Modeled completion time of a fixed cyclic peer rotation (Sec. 6.3, Table 3
 * "fixed peer rotation"), the baseline the demand-aware planner is compared
 * with, on the topology of `cat`: stage s = 1..N-1 pairs rank i with rank
 * (i + s) mod N and moves all of D_i,(i+s) (demand: host int64 [N, N]);
 * stages with no bytes are skipped.  path_rule VP_ROTATION_NEAREST_PATH puts
 * each lane on its pair's nearest path; VP_ROTATION_DYNAMIC_PATH lets every
 * stage pick, among each pair's paths (PXB or NIC between two switches of a
 * socket, SYS or NIC between sockets when enabled), the choice that
 * finishes the stage first.  Lanes on one directed
 * resource share its capacity equally (a stage need not be contention-free),
 * so a lane runs at min(path rate, capacity / sharers) over its resources;
 * a stage takes lambda_ns plus its slowest lane.  *num / *den is the exact
 * time in ns.  Host only.  More than 20 lanes with a path choice in one
 * stage is VP_ERR_UNSUPPORTED; a negative entry VP_ERR_INVALID_ARGUMENT. */
enum { VP_ROTATION_DYNAMIC_PATH = 0, VP_ROTATION_NEAREST_PATH = 1 };
vp_status vp_rotation_time(const vp_catalog* cat, const int64_t* demand, int32_t path_rule, int64_t lambda_ns,
                           int64_t* num, int64_t* den);

const char* vp_status_string(vp_status s);
const char* vp_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* VP_H_ */
