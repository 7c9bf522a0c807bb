// vp_pack: channel-ordered send buffers (Sec. 5 "Device-resident buffer
// layout").  For the steps in which this rank's lane carries bytes, in
// schedule order, the next x bytes of the stream to that step's destination
// are appended to the send buffer.
//
// Kernels
//   slices   only when the planner's buffer layout is not passed: one block;
//            after one round of global loads everything runs in LDS: step
//            offsets (exclusive scan of this rank's lane volumes) and each
//            step's offset inside its destination's stream (a stable
//            counting sort of the steps by destination -- per-wave ballot
//            ranks over contiguous chunks, one scan over destinations and
//            waves -- then a scan of the volumes in (destination, step)
//            order).
//   index    one workgroup per step (split over a few when steps are long).
//            With the planner's layout every step checks that its slice
//            starts where the previous step's ended, so the slices tile the
//            send buffer.  Rows: every packed unit is one copy of a token
//            row; its send unit goes to the entry of that (token, routing
//            slot), tagged with the call's generation, so the list is never
//            cleared.  Heads: one checked descriptor per step.
//   scatter  rows: one workgroup per (token, copy), XCD-aware so that all
//            copies of a token run on one XCD: a source row leaves HBM once
//            however many destinations it has, and the XCDs write
//            neighbouring tokens at any moment; launch shape by row size.
//   gather   heads: workgroups per (step, part); every 16-byte vector's
//            source address follows from the step's stream position (token
//            and head by multiply-high division), so no per-unit table is
//            written or read; non-temporal stores.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>

#include "internal.h"

namespace vp {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

__device__ inline void report(int32_t* status, int code) { atomicCAS(status, 0, code); }

__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Descriptor of one step in which this rank's lane carries units.
struct StepDesc {
  int64_t first;   // rows: index of the step's first unit in sorted_tok; heads: unit offset in the stream
  int32_t u0, nu;  // first send unit, unit count
  int32_t h0, h;   // heads: first head of the destination and its head count
};

struct SliceArgs {
  int mode;
  const int32_t *Kp, *dst;
  const int64_t* bytes;
  int32_t k_max, N, self;
  int64_t unit, T, send_capacity, token_stride;
  const int64_t* bounds;     // rows: dest_off [N+1] (units); heads: head_lo [N+1]
  int64_t* step_off;
  StepDesc* desc;            // carrying steps (any order)
  int32_t* n_desc;
  int32_t* status;
};

constexpr int kSliceWaves = 16;

// Dynamic LDS of the slice kernel for schedule capacity k_max and N ranks.
size_t slice_lds_bytes(int32_t k_max, int32_t N) {
  return (size_t)(N + 1) * 8 + (size_t)(2 * k_max + 1) * 4 + (size_t)kSliceWaves * N * 4 +
         (size_t)kSliceWaves * 64 * 4 + (size_t)k_max * 2 + 16;
}

// Inclusive scan over the 64 lanes of a wavefront.
__device__ inline int64_t wave_incl_scan(int64_t v, int lane) {
  for (int o = 1; o < 64; o <<= 1) {
    const int64_t y = __shfl_up(v, o);
    if (lane >= o) v += y;
  }
  return v;
}

__global__ void __launch_bounds__(1024) slices_kernel(SliceArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int N = a.N;
  int64_t* bo = (int64_t*)smem;                 // N+1: stream bounds (dest_off or head_lo)
  int32_t* so = (int32_t*)(bo + N + 1);         // k_max+1: units per step, then step offsets (units)
  int32_t* cl = so + a.k_max + 1;               // k_max: step offset inside its wave chunk's share of the stream
  int32_t* wv = cl + a.k_max;                   // [16][N]: per-wave units per destination, then prefixes
  int32_t* xl = wv + kSliceWaves * N;           // [16][64]: lane staging for match-group sums
  int16_t* jv = (int16_t*)(xl + kSliceWaves * 64);  // k_max: destination of step k, N when idle
  __shared__ int64_t wtot[kSliceWaves];
  __shared__ int32_t Ks, n_live;

  const int64_t cap_units = a.send_capacity / a.unit;
  if (tid == 0) {
    int K = *a.Kp;
    if (K < 0 || K > a.k_max) {
      report(a.status, VP_ERR_INVALID_ARGUMENT);
      K = 0;
    }
    // every head a destination owns must lie inside the token row
    if (a.mode == 1 && (a.bounds[0] < 0 || a.bounds[N] * a.unit > a.token_stride)) {
      report(a.status, VP_ERR_INVALID_ARGUMENT);
      K = 0;
    }
    Ks = K;
    n_live = 0;
    *a.n_desc = 0;
  }
  for (int i = tid; i < kSliceWaves * N; i += 1024) wv[i] = 0;
  for (int b = tid; b <= N; b += 1024) bo[b] = a.bounds[b];
  __syncthreads();
  const int K = Ks;
  // each thread owns E consecutive steps for the loads and the step scan
  const int E = (K + 1023) / 1024;
  const int k_beg = tid * E < K ? tid * E : K, k_end = k_beg + E < K ? k_beg + E : K;

  // 1. the only global loads of the schedule: this rank's lane per step
  int64_t mine = 0;
  for (int k = k_beg; k < k_end; ++k) {
    const int64_t x = a.bytes[(size_t)k * N + a.self];
    const int j = a.dst[(size_t)k * N + a.self];
    int b = N;
    int32_t u = 0;
    if (x != 0) {
      if (x < 0 || x % a.unit != 0 || j < 0 || j >= N || j == a.self) {
        report(a.status, VP_ERR_INVALID_ARGUMENT);
      } else if (x / a.unit > cap_units) {
        report(a.status, VP_ERR_CAPACITY);
      } else {
        b = j;
        u = (int32_t)(x / a.unit);
      }
    }
    so[k] = u;
    jv[k] = (int16_t)b;
    mine += u;
  }

  // 2. step offsets: exclusive scan of the units in schedule order
  const int64_t incl = wave_incl_scan(mine, lane);
  if (lane == 63) wtot[w] = incl;
  __syncthreads();
  int64_t run = incl - mine, total = 0;
  for (int v = 0; v < kSliceWaves; ++v) {
    if (v < w) run += wtot[v];
    total += wtot[v];
  }
  if (total > cap_units) {
    if (tid == 0) {
      report(a.status, VP_ERR_CAPACITY);
      a.step_off[K] = total * a.unit;
    }
    return;
  }
  for (int k = k_beg; k < k_end; ++k) {
    const int32_t u = so[k];
    so[k] = (int32_t)run;
    a.step_off[k] = run * a.unit;
    run += u;
  }
  if (tid == 0) {
    so[K] = (int32_t)total;
    a.step_off[K] = total * a.unit;
  }
  __syncthreads();

  // 3. offset of each step inside its destination's stream: the units of the
  //    earlier steps to the same destination.  Wave v walks the chunk
  //    [v*C, (v+1)*C) in order, keeping a running total per destination;
  //    lanes of one 64-step slice that share a destination (ballot match
  //    mask) add the units of the lower lanes of their group.
  const int C = (((K + kSliceWaves - 1) / kSliceWaves) + 63) & ~63;
  {
    int bits = 0;
    while ((1 << bits) < N) ++bits;
    const uint64_t lt = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    const uint64_t gt = lane == 63 ? 0ull : (~0ull << (lane + 1));
    int32_t* acc = wv + w * N;
    int32_t* stage = xl + w * 64;
    const int c_lo = w * C, c_hi = c_lo + C < K ? c_lo + C : K;
    for (int k0 = c_lo; k0 < c_hi; k0 += 64) {
      const int k = k0 + lane;
      const int b = k < c_hi ? jv[k] : N;
      const bool live = b < N;
      const int32_t u = live ? so[k + 1] - so[k] : 0;
      uint64_t same = __ballot(live);
      for (int bt = 0; bt < bits; ++bt) {
        const uint64_t ones = __ballot(live && ((b >> bt) & 1));
        same &= ((b >> bt) & 1) ? ones : ~ones;
      }
      stage[lane] = u;
      wave_sync();
      int32_t pre = 0;
      for (uint64_t m = same & lt; m; m &= m - 1) pre += stage[__builtin_ctzll(m)];
      const int32_t r = live ? acc[b] + pre : 0;
      wave_sync();
      if (live && (same & gt) == 0) acc[b] = r + u;
      wave_sync();
      if (live) cl[k] = r;
    }
  }
  __syncthreads();
  for (int b = tid; b < N; b += 1024) {
    int32_t s = 0;
    for (int v = 0; v < kSliceWaves; ++v) {
      const int32_t t = wv[v * N + b];
      wv[v * N + b] = s;
      s += t;
    }
  }
  __syncthreads();

  // 4. descriptors of the carrying steps; every slice must fit its stream
  for (int k = k_beg; k < k_end; ++k) {
    const int b = jv[k];
    if (b == N) continue;
    const int64_t c = (int64_t)cl[k] + wv[(k / C) * N + b];
    const int32_t u = so[k + 1] - so[k];
    const int64_t h = bo[b + 1] - bo[b];
    const int64_t len = a.mode == 0 ? h : a.T * h;
    if (c + u > len) {
      report(a.status, VP_ERR_INVALID_ARGUMENT);
      continue;
    }
    StepDesc d;
    d.first = a.mode == 0 ? bo[b] + c : c;
    d.u0 = so[k];
    d.nu = u;
    d.h0 = a.mode == 0 ? 0 : (int32_t)bo[b];
    d.h = a.mode == 0 ? 0 : (int32_t)h;
    a.desc[atomicAdd(&n_live, 1)] = d;
  }
  __syncthreads();
  if (tid == 0) *a.n_desc = n_live;
}

struct IndexArgs {
  int mode, k, self, N, k_max;
  int64_t unit, T, token_stride, send_capacity;
  uint32_t gen;                // this call's generation of the copy counters
  const int32_t* sorted_tok;
  const uint8_t* sorted_slot;
  const StepDesc* desc;        // descriptors from the slice kernel, or
  int32_t* n_desc;
  const int32_t *Kp, *dst;     // the schedule and the planner's buffer layout
  const int64_t *bytes, *send_off, *stream_off;
  const int64_t* bounds;       // rows: dest_off; heads: head_lo
  int64_t* step_off;
  uint32_t* hdr;               // [0]: generation, read by the scatter; bytes 8..15: token stride
  unsigned long long* lst;     // rows: [T][k] generation << 32 | send unit of each routing slot
  StepDesc* hdesc;             // heads with the planner's layout: one descriptor per step
  int32_t* status;
};

constexpr int kIndexThreads = 256;

// One workgroup per step.  With the planner's buffer layout the workgroup
// derives its step's descriptor itself (step offsets, checks); otherwise it
// takes the slice kernel's.  The layout must tile the send buffer: step k's
// slice starts where step k-1's ended (step 0's at 0), which each workgroup
// checks against its predecessor, so by induction the send offsets are the
// running sum of this rank's lane volumes.  Rows: every packed unit is one
// (token, routing slot) assignment; its send unit goes to that slot's entry,
// tagged with the call's generation (strictly increasing), so the entries of
// slots this call does not pack (local experts, streams not covered) are
// recognisably old and the list is never cleared.  Heads: the step's checked
// descriptor (no units when the lane is idle); the gather reads only
// descriptors of this call, and none when a step failed its checks.
__global__ void __launch_bounds__(kIndexThreads) index_kernel(IndexArgs a) {
  // workgroup (i, y) handles part y of step i's units (gridDim.y parts)
  const int i = blockIdx.x, tid = threadIdx.x, y = blockIdx.y, ny = gridDim.y;
  const bool lead = y == 0 && tid == 0;   // the one thread that writes a step's offsets
  if (i == 0 && lead) {
    *a.hdr = a.gen;
    *(int64_t*)(a.hdr + 2) = a.token_stride;
  }
  StepDesc d;
  if (a.send_off) {
    const int K = *a.Kp, st = *a.status;
    if (K < 0 || K > a.k_max) {
      if (i == 0 && lead) {
        report(a.status, VP_ERR_INVALID_ARGUMENT);
        if (a.mode == 1) *a.n_desc = 0;
      }
      return;
    }
    if (i == 0 && lead) {
      if (a.mode == 1) *a.n_desc = K;
      if (K == 0) a.step_off[0] = 0;
    }
    if (st != 0 || i >= K) return;
    const size_t o = (size_t)i * a.N + a.self;
    const int64_t x = a.bytes[o], so = a.send_off[o], co = a.stream_off[o];
    const int j = a.dst[o];
    const int64_t prev_end = i == 0 ? 0 : a.send_off[o - a.N] + a.bytes[o - a.N];
    d.first = 0;
    d.u0 = 0;
    d.nu = 0;
    d.h0 = 0;
    d.h = 1;
    bool ok = so == prev_end;
    if (lead) {
      a.step_off[i] = so;
      if (i == K - 1) a.step_off[K] = so + x;
    }
    if (ok && x != 0) {
      ok = x > 0 && x % a.unit == 0 && so >= 0 && so % a.unit == 0 && co >= 0 && co % a.unit == 0 &&
           j >= 0 && j < a.N && j != a.self;
      if (ok && so + x > a.send_capacity) {
        if (lead) report(a.status, VP_ERR_CAPACITY);
        return;
      }
      int64_t h = 0, b0 = 0;
      if (ok) {
        b0 = a.bounds[j];
        h = a.bounds[j + 1] - b0;
        // heads: every head of the destination lies inside the token row
        if (a.mode == 1) ok = b0 >= 0 && h >= 1 && (b0 + h) * a.unit <= a.token_stride;
        ok = ok && co + x <= (a.mode == 0 ? h : a.T * h) * a.unit;
      }
      if (ok) {
        d.first = a.mode == 0 ? b0 + co / a.unit : co / a.unit;
        d.u0 = (int32_t)(so / a.unit);
        d.nu = (int32_t)(x / a.unit);
        d.h0 = a.mode == 0 ? 0 : (int32_t)b0;
        d.h = a.mode == 0 ? 0 : (int32_t)h;
      }
    }
    if (!ok) {
      if (lead) report(a.status, VP_ERR_INVALID_ARGUMENT);
      return;
    }
    if (a.mode == 1) {
      if (lead) a.hdesc[i] = d;
      return;
    }
    if (d.nu == 0) return;
  } else {
    if (a.mode == 1) return;   // the slice kernel wrote the descriptors
    const int n = *a.n_desc, st = *a.status;
    if (i >= n || st != 0) return;
    d = a.desc[i];
  }
  const unsigned long long g = (unsigned long long)a.gen << 32;
  for (int u = tid + y * kIndexThreads; u < d.nu; u += kIndexThreads * ny) {
    const int64_t tok = a.sorted_tok[d.first + u];
    const int slot = a.sorted_slot[d.first + u];
    if (tok < 0 || tok >= a.T || slot >= a.k) {
      report(a.status, VP_ERR_INVALID_ARGUMENT);
      continue;
    }
    a.lst[tok * a.k + slot] = g | (unsigned)(d.u0 + u);
  }
}

// Rows: one workgroup per (token, copy slot).  Workgroups are handed to the
// eight XCDs round-robin; the mapping below gives XCD x the tokens t with
// t % 8 == x, all copy slots of a token back to back, so a token's copies
// are read on one XCD in a row (the row leaves HBM once, the repeats hit
// that XCD's L2) while the eight XCDs work on neighbouring tokens, whose
// copies land next to each other in every destination's stream.  TH threads
// move the row in passes of V 16-byte vectors per thread: all V loads of a
// pass are issued before its first store, so a wavefront keeps V KiB in
// flight.
template <int TH, int V>
__global__ void __launch_bounds__(TH) scatter_rows_kernel(
    const unsigned char* __restrict__ src, const unsigned long long* __restrict__ lst,
    const uint32_t* __restrict__ hdr, int64_t T, int k, int64_t unit, int64_t vpu,
    unsigned char* __restrict__ send, const int32_t* status) {
  const int64_t idx = blockIdx.x >> 3;
  const int64_t t = (idx / k) * 8 + (blockIdx.x & 7);
  const int c = (int)(idx % k);
  if (*status != 0 || t >= T) return;
  // this workgroup stores the token's c-th copy in send order (not routing
  // order), so the copies the eight XCDs store at one time sit in nearby
  // steps of the send buffer.  Every wavefront ranks the token's entries
  // itself (one 64-lane load, k shuffles); more than 64 slots keep routing
  // order.
  const uint32_t gen = *hdr;
  const int lane = threadIdx.x & 63;
  uint32_t u;
  if (k <= 64) {
    const unsigned long long ei = lane < k ? lst[t * k + lane] : 0;
    const bool ok = lane < k && (uint32_t)(ei >> 32) == gen;
    const uint32_t ui = ok ? (uint32_t)ei : 0xFFFFFFFFu;
    int below = 0;
    for (int j = 0; j < k; ++j) below += (uint32_t)__shfl((int)ui, j) < ui;
    const unsigned long long m = __ballot(ok && below == c);
    if (m == 0) return;   // fewer than c + 1 copies of this token are packed by this call
    u = (uint32_t)__shfl((int)ui, __builtin_ctzll(m));
  } else {
    const unsigned long long e = lst[t * k + c];
    if ((uint32_t)(e >> 32) != gen) return;
    u = (uint32_t)e;
  }
  const u32x4* row = (const u32x4*)(src + t * unit);
  u32x4* d = (u32x4*)(send + (int64_t)u * unit);
  for (int64_t e0 = threadIdx.x; e0 < vpu; e0 += (int64_t)V * TH) {
    u32x4 r[V];
#pragma unroll
    for (int i = 0; i < V; ++i)
      if (e0 + i * TH < vpu) r[i] = row[e0 + i * TH];
#pragma unroll
    for (int i = 0; i < V; ++i)
      if (e0 + i * TH < vpu) __builtin_nontemporal_store(r[i], d + e0 + i * TH);
  }
}

constexpr int kGatherThreads = 256;
constexpr int kGatherUnroll = 4;

// Heads: workgroup (i, y) copies part y of descriptor i's units.  A step's
// slice is stream positions first .. first+nu-1 of its destination, which
// owns heads h0 .. h0+h-1 of every token: position p is token p / h, head
// h0 + p % h.  Divisions are multiply-high by ceil(2^48 / divisor), exact
// for dividends below 2^48 / divisor (the host bounds T * heads^2 and the
// send vectors).  Every vector's source is checked against the activations
// before it is loaded.  All loads of a pass are issued before its stores.
__global__ void __launch_bounds__(kGatherThreads) gather_heads_kernel(
    const unsigned char* __restrict__ src, const StepDesc* __restrict__ desc, const int32_t* n_desc,
    const uint32_t* hdr, int64_t T, int64_t unit, int64_t vpu, uint64_t vpu_magic, int64_t cap_units,
    unsigned char* __restrict__ send, int32_t* status) {
  const int i = blockIdx.x;
  if (*status != 0 || i >= *n_desc) return;
  const StepDesc d = desc[i];
  if (d.nu <= 0) return;
  const int64_t token_stride = *(const int64_t*)(hdr + 2);
  if (d.h < 1 || d.h0 < 0 || ((int64_t)d.h0 + d.h) * unit > token_stride || d.u0 < 0 ||
      (int64_t)d.u0 + d.nu > cap_units || d.first < 0 || d.first + d.nu > T * d.h) {
    if (threadIdx.x == 0 && blockIdx.y == 0) report(status, VP_ERR_INVALID_ARGUMENT);
    return;
  }
  const uint64_t h_magic = ((uint64_t(1) << 48) + (uint64_t)d.h - 1) / (uint64_t)d.h;
  const int64_t nvec = (int64_t)d.nu * vpu;
  const int64_t stride = (int64_t)gridDim.y * kGatherThreads;
  unsigned char* out = send + (int64_t)d.u0 * unit;
  const unsigned char* base = src + (int64_t)d.h0 * unit;
  for (int64_t v = (int64_t)blockIdx.y * kGatherThreads + threadIdx.x; v < nvec; v += kGatherUnroll * stride) {
    u32x4 r[kGatherUnroll];
#pragma unroll
    for (int m = 0; m < kGatherUnroll; ++m) {
      const int64_t vv = v + m * stride;
      if (vv < nvec) {
        const int64_t u = (int64_t)__umul64hi((uint64_t)vv << 16, vpu_magic);
        const int64_t in = vv - u * vpu;
        const int64_t p = d.first + u;
        const int64_t tok = (int64_t)__umul64hi((uint64_t)p << 16, h_magic);
        const int64_t hd = p - tok * d.h;
        r[m] = *(const u32x4*)(base + tok * token_stride + hd * unit + in * 16);
      }
    }
#pragma unroll
    for (int m = 0; m < kGatherUnroll; ++m) {
      const int64_t vv = v + m * stride;
      if (vv < nvec) __builtin_nontemporal_store(r[m], (u32x4*)(out + vv * 16));
    }
  }
}

size_t desc_bytes(int32_t k_max) { return align_up((size_t)k_max * sizeof(StepDesc) + 16, 256); }

constexpr size_t kHeader = 256;   // [0]: the generation of the last prepare

}  // namespace

size_t pack_workspace(int32_t k_max, int64_t send_capacity, int64_t unit, int64_t T, int32_t k) {
  (void)send_capacity;
  (void)unit;
  const size_t head = kHeader + desc_bytes(k_max);
  if (k > 0) return head + (size_t)T * (size_t)k * 8;
  return head;
}

namespace {
std::atomic<uint32_t> g_generation{0};
}

vp_status launch_pack(const PackLaunch& a, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const size_t lds = slice_lds_bytes(a.k_max, a.N);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return set_error(VP_ERR_HIP, "hipGetDevice failed");
  int lds_max = 0;
  if (hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
    return set_error(VP_ERR_HIP, "hipDeviceGetAttribute failed");
  const bool layout = a.send_off != nullptr;
  if (!layout && lds + 1024 > (size_t)lds_max)
    return set_error(VP_ERR_UNSUPPORTED, "k_max too large for the slice table");
  if (a.unit % 16 != 0) return set_error(VP_ERR_INVALID_ARGUMENT, "unit must be a multiple of 16");
  if ((a.mode == 0) != (a.k > 0)) return set_error(VP_ERR_INVALID_ARGUMENT, "top-k must be > 0 exactly for rows");
  // unit counts and send-unit indices are held in 32 bits
  if (a.send_capacity / a.unit >= ((int64_t)1 << 31)) return set_error(VP_ERR_UNSUPPORTED, "send buffer too large");
  char* ws = (char*)a.ws;
  uint32_t* hdr = (uint32_t*)ws;
  StepDesc* desc = (StepDesc*)(ws + kHeader);
  int32_t* n_desc = (int32_t*)(ws + kHeader + (size_t)a.k_max * sizeof(StepDesc));
  char* rest = ws + kHeader + desc_bytes(a.k_max);
  unsigned long long* lst = (unsigned long long*)rest;
  // heads: positions are below T * heads per token and are divided by at
  // most that many heads in the gather; both stay within the division's range
  if (a.mode == 1) {
    const int64_t hmax = a.token_stride / a.unit;
    if (a.T > 0 && (hmax > ((int64_t)1 << 15) || a.T > (((int64_t)1 << 47) / hmax) / hmax))
      return set_error(VP_ERR_UNSUPPORTED, "too many heads per token for this many tokens");
  }

  if (a.stages & 1) {
    uint32_t gen = ++g_generation;
    if (gen == 0) gen = ++g_generation;   // zero is the value of a cleared workspace
    if (!layout) {
      SliceArgs sa{a.mode, a.K, a.dst, a.bytes, a.k_max, a.N, a.self_rank, a.unit, a.T, a.send_capacity,
                   a.token_stride, a.mode == 0 ? a.dest_off : a.head_lo, a.step_off, desc, n_desc, a.status};
      if (hipFuncSetAttribute((const void*)slices_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)lds) != hipSuccess)
        return set_error(VP_ERR_HIP, "cannot raise the slice kernel's LDS limit");
      hipLaunchKernelGGL(slices_kernel, dim3(1), dim3(1024), lds, s, sa);
    }
    IndexArgs ia{a.mode, a.k, a.self_rank, a.N, a.k_max, a.unit, a.T, a.token_stride, a.send_capacity, gen,
                 a.sorted_tok, a.sorted_slot, desc, n_desc, a.K, a.dst, a.bytes, a.send_off, a.stream_off,
                 a.mode == 0 ? a.dest_off : a.head_lo, a.step_off, hdr, lst, desc, a.status};
    // rows: a step holds up to one destination's whole stream: split it over
    // up to 16 workgroups so that a thread handles about two of its units;
    // heads: one thread per step does all the work
    const int64_t units = a.mode == 0 ? a.T * a.k : 0;
    const int64_t per_step = (units + a.N - 1) / std::max(1, a.N);
    const int ny = (int)std::min<int64_t>(16, std::max<int64_t>(1, (per_step + 2 * kIndexThreads - 1) /
                                                                      (2 * kIndexThreads)));
    hipLaunchKernelGGL(index_kernel, dim3(a.k_max, ny), dim3(kIndexThreads), 0, s, ia);
  }
  if (!(a.stages & 2)) {
    if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "pack launch failed");
    return VP_OK;
  }
  const int64_t vpu = a.unit / 16;
  if (a.mode == 0) {
    const int64_t blocks = (a.T + 7) / 8 * 8 * a.k;
    if (blocks > 0) {
      if (blocks >= ((int64_t)1 << 31)) return set_error(VP_ERR_UNSUPPORTED, "too many token copies");
      const unsigned char* sp = (const unsigned char*)a.src;
      unsigned char* dp = (unsigned char*)a.send;
      const dim3 grid((unsigned)blocks);
      // about 2 KiB per wavefront: rows up to 2, 4 and 8 KiB take 1, 2 and 4
      // wavefronts of two vectors per thread; longer rows take 8 wavefronts
      // with one vector per thread per pass (measured best on 4, 8 and 14 KiB
      // rows)
      if (vpu <= 128)
        hipLaunchKernelGGL((scatter_rows_kernel<64, 2>), grid, dim3(64), 0, s, sp, lst, hdr, a.T, a.k, a.unit, vpu,
                           dp, a.status);
      else if (vpu <= 256)
        hipLaunchKernelGGL((scatter_rows_kernel<128, 2>), grid, dim3(128), 0, s, sp, lst, hdr, a.T, a.k, a.unit,
                           vpu, dp, a.status);
      else if (vpu <= 512)
        hipLaunchKernelGGL((scatter_rows_kernel<256, 2>), grid, dim3(256), 0, s, sp, lst, hdr, a.T, a.k, a.unit,
                           vpu, dp, a.status);
      else
        hipLaunchKernelGGL((scatter_rows_kernel<512, 1>), grid, dim3(512), 0, s, sp, lst, hdr, a.T, a.k, a.unit,
                           vpu, dp, a.status);
    }
  } else {
    // u = floor(v / vpu) = mulhi(v << 16, ceil(2^48 / vpu)) for v < 2^48 / vpu
    const unsigned __int128 two48 = (unsigned __int128)1 << 48;
    const uint64_t magic = (uint64_t)((two48 + (unsigned __int128)vpu - 1) / (unsigned __int128)vpu);
    const int64_t max_vec = a.send_capacity / 16;
    if (max_vec >= ((int64_t)1 << 48) / vpu) return set_error(VP_ERR_UNSUPPORTED, "send buffer too large");
    // parts per step: about 16 KiB each for an average step of k_max
    const int64_t per_step = a.send_capacity / std::max(1, a.k_max);
    const int ny = (int)std::min<int64_t>(64, std::max<int64_t>(1, (per_step + 16383) / 16384));
    hipLaunchKernelGGL(gather_heads_kernel, dim3((unsigned)a.k_max, (unsigned)ny), dim3(kGatherThreads), 0, s,
                       (const unsigned char*)a.src, desc, n_desc, hdr, a.T, a.unit, vpu, magic,
                       a.send_capacity / a.unit, (unsigned char*)a.send, a.status);
  }
  if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "pack launch failed");
  return VP_OK;
}

}  // namespace vp
