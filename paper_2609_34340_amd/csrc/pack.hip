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
//            order).  It writes one descriptor per step, in step order.
//   index    rows: one workgroup per step (split over a few when steps are
//            long).  With the planner's layout every step checks that its
//            slice starts where the previous step's ended, so the slices
//            tile the send buffer.  Every packed unit is one copy of a token
//            row; its send unit goes to the entry of that (token, routing
//            slot), tagged with the call's generation, so the list is never
//            cleared.  Heads with the planner's layout: one thread per step
//            checks the step the same way and writes its descriptor.
//   scatter  rows: one workgroup per (token, copy), XCD-aware so that all
//            copies of a token run on one XCD: a source row leaves HBM once
//            however many destinations it has, and the XCDs write
//            neighbouring tokens at any moment; launch shape by row size.
//   gather   heads: the send buffer is cut into equal contiguous ranges, one
//            per workgroup, whatever the step sizes; a workgroup finds the
//            step holding its first unit by a parallel search over the step
//            descriptors and walks the steps of its range.  Source addresses
//            follow from the step's stream position (token and head), with
//            the divisions done once per range and then carried forward in
//            32 bits, so no per-unit table is written or read; non-temporal
//            stores.
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
  uint64_t h_m40;  // heads: ceil(2^40 / h), for the gather's 32-bit divisions by h
  uint64_t h_m64;  // heads: ceil(2^64 / h), 0 for h = 1, for its 64-bit ones
};

// floor(x / d) for 0 <= x < 2^53 and 1 <= d < 2^53, without a 64-bit
// integer division: the correctly rounded double quotient is within one of
// it (below 2^52), and one step against the integer remainder makes it
// exact.  Callers that cannot bound x check q * d against x.
__host__ __device__ inline int64_t fdiv53(int64_t x, int64_t d) {
  int64_t q = (int64_t)((double)x / (double)d);
  const int64_t r = x - q * d;
  if (r < 0)
    --q;
  else if (r >= d)
    ++q;
  return q;
}

// Multiply-high reciprocals of a divisor 1 <= d < 2^20 (see StepDesc):
// ceil(2^40 / d), and ceil(2^64 / d) = 2^24 floor(2^40 / d) + the rest,
// 0 for d = 1.
__host__ __device__ inline uint64_t magic40(uint64_t d) {
  const int64_t q = fdiv53((int64_t)1 << 40, (int64_t)d);
  return (uint64_t)q + ((uint64_t)q * d != (uint64_t(1) << 40));
}
__host__ __device__ inline uint64_t magic64(uint64_t d) {
  if (d == 1) return 0;
  const int64_t q40 = fdiv53((int64_t)1 << 40, (int64_t)d);
  const int64_t r40 = ((int64_t)1 << 40) - q40 * (int64_t)d;
  const int64_t t = fdiv53(r40 << 24, (int64_t)d);
  return ((uint64_t)q40 << 24) + (uint64_t)t + ((r40 << 24) != t * (int64_t)d);
}

// floor(x / d) from m = magic64(d): x * m / 2^64 = x / d + x * e / (d 2^64)
// with e = m d - 2^64 < d, exact for x * d < 2^64.
__device__ inline uint64_t div64(uint64_t x, uint64_t m) { return m == 0 ? x : __umul64hi(x, m); }

// Head of the pack workspace.  The rows scatter reads the generation; the
// heads gather reads the rest, written by the prepare stage.
struct PackHeader {
  uint32_t gen;          // generation of the last rows prepare
  int32_t n_steps;       // heads: K of the last prepare (0 for a refused K)
  int64_t token_stride;  // heads: bytes per token row of the activations
  int64_t units;         // heads: send units of the last prepare
};

struct SliceArgs {
  int mode;
  const int32_t *Kp, *dst;
  const int64_t* bytes;
  int32_t k_max, N, self;
  int64_t unit, T, send_capacity, token_stride;
  const int64_t* bounds;     // rows: dest_off [N+1] (units); heads: head_lo [N+1]
  int64_t* step_off;
  StepDesc* desc;            // one per step, in step order
  int32_t* u0s;              // the descriptors' first units, apart
  int32_t* n_desc;
  PackHeader* hdr;           // heads: step count, token stride, send units
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
  __shared__ int32_t Ks;

  const int64_t cap_units = a.send_capacity / a.unit;
  if (tid == 0) {
    int K = *a.Kp;
    if (K < 0 || K > a.k_max) {
      report(a.status, VP_ERR_INVALID_ARGUMENT);
      K = 0;
    }
    // every head a destination owns must lie inside the token row
    if (a.mode == 1 && (a.bounds[0] < 0 || a.bounds[N] > a.token_stride / a.unit)) {
      report(a.status, VP_ERR_INVALID_ARGUMENT);
      K = 0;
    }
    Ks = K;
    *a.n_desc = 0;
    if (a.mode == 1) {
      a.hdr->n_steps = K;
      a.hdr->token_stride = a.token_stride;
    }
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
    if (a.mode == 1) a.hdr->units = total;
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

  // 4. one descriptor per step, in step order (idle steps carry no units
  //    and start where the next step starts); every slice must fit its
  //    stream
  for (int k = k_beg; k < k_end; ++k) {
    const int b = jv[k];
    StepDesc d;
    d.first = 0;
    d.u0 = so[k];
    d.nu = 0;
    d.h0 = 0;
    d.h = a.mode == 0 ? 0 : 1;
    if (b != N) {
      const int64_t c = (int64_t)cl[k] + wv[(k / C) * N + b];
      const int32_t u = so[k + 1] - so[k];
      const int64_t h = bo[b + 1] - bo[b];
      const int64_t len = a.mode == 0 ? h : a.T * h;
      // heads: the destination's heads lie inside the token row
      const bool heads_ok = a.mode == 0 || (bo[b] >= 0 && h >= 1 && bo[b + 1] <= a.token_stride / a.unit);
      if (!heads_ok || c + u > len) report(a.status, VP_ERR_INVALID_ARGUMENT);
      d.first = a.mode == 0 ? bo[b] + c : c;
      d.nu = u;
      d.h0 = a.mode == 0 ? 0 : (int32_t)bo[b];
      d.h = a.mode == 0 ? 0 : (int32_t)h;
    }
    d.h_m40 = d.h >= 1 ? magic40((uint64_t)d.h) : 0;
    d.h_m64 = d.h >= 1 ? magic64((uint64_t)d.h) : 0;
    a.desc[k] = d;
    a.u0s[k] = d.u0;
  }
  __syncthreads();
  if (tid == 0) *a.n_desc = K;
}

struct IndexArgs {
  int mode, k, self, N, k_max;
  int64_t unit, T, token_stride, send_capacity;
  int64_t heads_per_row;       // heads: token_stride / unit
  uint32_t gen;                // this call's generation of the copy counters
  const int32_t* sorted_tok;
  const uint8_t* sorted_slot;
  StepDesc* desc;              // rows: the slice kernel's descriptors; heads: written here
  int32_t* u0s;                // heads: the descriptors' first units, apart
  int32_t* n_desc;
  const int32_t *Kp, *dst;     // the schedule and the planner's buffer layout
  const int64_t *bytes, *send_off, *stream_off;
  const int64_t* bounds;       // rows: dest_off; heads: head_lo
  int64_t* step_off;
  PackHeader* hdr;
  unsigned long long* lst;     // rows: [T][k] generation << 32 | send unit of each routing slot
  int32_t* status;
};

constexpr int kIndexThreads = 256;

// Rows: one workgroup per step.  With the planner's buffer layout the
// workgroup derives its step's slice itself (step offsets, checks);
// otherwise it takes the slice kernel's descriptor.  The layout must tile
// the send buffer: step k's slice starts where step k-1's ended (step 0's at
// 0), which each workgroup checks against its predecessor, so by induction
// the send offsets are the running sum of this rank's lane volumes.  Every
// packed unit is one (token, routing slot) assignment; its send unit goes to
// that slot's entry, tagged with the call's generation (strictly
// increasing), so the entries of slots this call does not pack (local
// experts, streams not covered) are recognisably old and the list is never
// cleared.
__global__ void __launch_bounds__(kIndexThreads) index_kernel(IndexArgs a) {
  // workgroup (i, y) handles part y of step i's units (gridDim.y parts)
  const int i = blockIdx.x, tid = threadIdx.x, y = blockIdx.y, ny = gridDim.y;
  const bool lead = y == 0 && tid == 0;   // the one thread that writes a step's offsets
  if (i == 0 && lead) a.hdr->gen = a.gen;
  StepDesc d;
  if (a.send_off) {
    const int K = *a.Kp, st = *a.status;
    if (K < 0 || K > a.k_max) {
      if (i == 0 && lead) report(a.status, VP_ERR_INVALID_ARGUMENT);
      return;
    }
    if (i == 0 && lead && K == 0) a.step_off[0] = 0;
    if (st != 0 || i >= K) return;
    const size_t o = (size_t)i * a.N + a.self;
    const int64_t x = a.bytes[o], so = a.send_off[o], co = a.stream_off[o];
    const int j = a.dst[o];
    const int64_t prev_end = i == 0 ? 0 : a.send_off[o - a.N] + a.bytes[o - a.N];
    bool ok = so == prev_end;
    if (lead) {
      a.step_off[i] = so;
      if (i == K - 1) a.step_off[K] = so + x;
    }
    d.nu = 0;
    if (ok && x != 0) {
      ok = x > 0 && x % a.unit == 0 && so >= 0 && so % a.unit == 0 && co >= 0 && co % a.unit == 0 &&
           j >= 0 && j < a.N && j != a.self;
      if (ok && so + x > a.send_capacity) {
        if (lead) report(a.status, VP_ERR_CAPACITY);
        return;
      }
      if (ok) {
        const int64_t b0 = a.bounds[j], h = a.bounds[j + 1] - b0;
        ok = co + x <= h * a.unit;
        d.first = b0 + co / a.unit;
        d.u0 = (int32_t)(so / a.unit);
        d.nu = (int32_t)(x / a.unit);
      }
    }
    if (!ok) {
      if (lead) report(a.status, VP_ERR_INVALID_ARGUMENT);
      return;
    }
    if (d.nu == 0) return;
  } else {
    const int n = *a.n_desc, st = *a.status;
    if (i >= n || st != 0) return;
    d = a.desc[i];
    if (d.nu == 0) return;
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

// Step i of a heads schedule with the planner's layout, as the rows index
// checks it (tiling, whole units, destination, stream bounds, capacity)
// plus that every head of the destination lies inside the token row; fills
// the step's descriptor (an idle step: no units, at its send offset, so the
// descriptors' first units ascend).  Returns 0, VP_ERR_INVALID_ARGUMENT or
// VP_ERR_CAPACITY.  hl(b) reads head_lo[b].
struct HeadsStep {
  int64_t x, so, co, prev_end;   // lane bytes, send offset, stream offset, end of step i-1's slice
  int j;                         // destination
};

template <class HeadLo>
__device__ inline int heads_step_desc(const HeadsStep& st, HeadLo hl, int N, int self, int64_t unit, int64_t T,
                                      int64_t heads_per_row, int64_t send_capacity, StepDesc& d) {
  d.first = 0;
  d.u0 = 0;
  d.nu = 0;
  d.h0 = 0;
  d.h = 1;
  d.h_m40 = uint64_t(1) << 40;
  d.h_m64 = 0;
  // whole units, checked by multiplying back (so any quotient is exact)
  const int64_t su = st.so >= 0 ? fdiv53(st.so, unit) : -1;
  if (st.so != st.prev_end || su < 0 || su * unit != st.so) return VP_ERR_INVALID_ARGUMENT;
  d.u0 = (int32_t)su;
  if (st.x == 0) return 0;
  const int64_t xu = st.x > 0 ? fdiv53(st.x, unit) : -1;
  const int64_t cu = st.co >= 0 ? fdiv53(st.co, unit) : -1;
  if (xu <= 0 || xu * unit != st.x || cu < 0 || cu * unit != st.co || st.j < 0 || st.j >= N || st.j == self)
    return VP_ERR_INVALID_ARGUMENT;
  if (st.so + st.x > send_capacity) return VP_ERR_CAPACITY;
  const int64_t b0 = hl(st.j), h = hl(st.j + 1) - b0;
  if (!(b0 >= 0 && h >= 1 && b0 + h <= heads_per_row && cu + xu <= T * h)) return VP_ERR_INVALID_ARGUMENT;
  d.first = cu;
  d.nu = (int32_t)xu;
  d.h0 = (int32_t)b0;
  d.h = (int32_t)h;
  d.h_m40 = magic40((uint64_t)h);
  d.h_m64 = magic64((uint64_t)h);
  return 0;
}

// Heads with the planner's layout: thread i checks step i and writes its
// descriptor; every step below K gets one.  The schedule arrays have k_max
// rows and head_lo is staged in LDS (up to 1024 ranks), so all of a step's
// loads are issued at once, before K is known.
constexpr int kHeadLoLds = 1025;

__global__ void __launch_bounds__(kIndexThreads) heads_index_kernel(IndexArgs a) {
  __shared__ int64_t hls[kHeadLoLds];
  const int i = blockIdx.x * kIndexThreads + threadIdx.x;
  const bool in = i < a.k_max;
  const bool staged = a.N + 1 <= kHeadLoLds;
  const size_t o = (size_t)i * a.N + a.self;
  HeadsStep st{0, 0, 0, 0, 0};
  if (in) {
    st.x = a.bytes[o];
    st.so = a.send_off[o];
    st.co = a.stream_off[o];
    st.j = a.dst[o];
    if (i > 0) st.prev_end = a.send_off[o - a.N] + a.bytes[o - a.N];
  }
  if (staged)
    for (int b = threadIdx.x; b <= a.N; b += kIndexThreads) hls[b] = a.bounds[b];
  const int K = *a.Kp, stat = *a.status;
  const bool bad_k = K < 0 || K > a.k_max;
  if (i == 0) {
    a.hdr->n_steps = bad_k ? 0 : K;
    a.hdr->token_stride = a.token_stride;
    if (bad_k) report(a.status, VP_ERR_INVALID_ARGUMENT);
    if (K == 0) {
      a.step_off[0] = 0;
      a.hdr->units = 0;
    }
  }
  __syncthreads();
  if (bad_k || stat != 0 || i >= K) return;
  a.step_off[i] = st.so;
  if (i == K - 1) {
    a.step_off[K] = st.so + st.x;
    a.hdr->units = (st.so + st.x) / a.unit;
  }
  StepDesc d;
  const int err = heads_step_desc(
      st, [&](int b) { return staged ? hls[b] : a.bounds[b]; }, a.N, a.self, a.unit, a.T, a.heads_per_row,
      a.send_capacity, d);
  if (err != 0) {
    report(a.status, err);
    return;
  }
  a.desc[i] = d;
  a.u0s[i] = d.u0;
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
    const PackHeader* __restrict__ hdr, int64_t T, int k, int64_t unit, int64_t vpu,
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
  const uint32_t gen = hdr->gen;
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
constexpr int kGatherPass = kGatherThreads * kGatherUnroll;   // vectors per pass of a workgroup

// floor(x / d) for x, d < 2^20: multiply-high by m = ceil(2^40 / d), exact
// because x * (m * d - 2^40) < x * d < 2^40.
__device__ inline uint32_t small_div(uint32_t x, uint64_t m) { return (uint32_t)(((uint64_t)x * m) >> 40); }

// Copies vectors [a, b) of the send buffer, which lie in the step of the
// checked descriptor d whose vectors start at sv0.  Stream position p is
// token p / h, head h0 + p % h; the unit and the (token, head) of a pass's
// first vector are divided out in 64 bits, a thread's offset from there
// (below 2^20 vectors) in 32 bits, all by multiply-high with the
// descriptor's reciprocals.  All loads of a pass are issued before its
// stores; lanes past the end copy the pass's last vector again (the same
// bytes to the same place), so neither carries branches.
template <int TH>
__device__ inline void copy_heads_range(const unsigned char* __restrict__ src, unsigned char* __restrict__ send,
                                        const StepDesc& d, int64_t a, int64_t b, int64_t sv0, int32_t vpu,
                                        uint64_t vpu_m40, uint64_t vpu_m64, int64_t unit, int64_t token_stride,
                                        int tid) {
  constexpr int kPass = TH * kGatherUnroll;
  const uint32_t h32 = (uint32_t)__builtin_amdgcn_readfirstlane(d.h);
  const uint64_t h_m40 = d.h_m40, h_m64 = d.h_m64;
  const uint32_t stride32 = (uint32_t)token_stride, unit32 = (uint32_t)unit;
  // vector a is vector r0 of unit q0 of the step; that unit is stream
  // position first + q0: token tok0, head hd0 of the destination's heads
  const int64_t q0 = (int64_t)div64((uint64_t)(a - sv0), vpu_m64);
  uint32_t r0 = (uint32_t)(a - sv0 - q0 * vpu);
  const int64_t p0 = d.first + q0;
  const int64_t tok0 = (int64_t)div64((uint64_t)p0, h_m64);
  uint32_t hd0 = (uint32_t)(p0 - tok0 * h32);
  const unsigned char* row = src + (int64_t)d.h0 * unit + tok0 * token_stride;   // token tok0's first head
  u32x4* out = (u32x4*)(send + a * 16);
  const int64_t n = b - a;
  for (int64_t e0 = 0; e0 < n; e0 += kPass) {
    const int64_t left = n - e0;
    const int last = left < kPass ? (int)left - 1 : kPass - 1;
    const unsigned char* at[kGatherUnroll];
    int es[kGatherUnroll];
#pragma unroll
    for (int m = 0; m < kGatherUnroll; ++m) {
      const int e = m * TH + tid < last ? m * TH + tid : last;
      es[m] = e;
      const uint32_t x = r0 + (uint32_t)e;
      const uint32_t du = small_div(x, vpu_m40);
      const uint32_t in = x - du * (uint32_t)vpu;
      const uint32_t hq = hd0 + du;
      const uint32_t dt = small_div(hq, h_m40);
      const uint32_t off = (hq - dt * h32) * unit32 + in * 16;   // inside the token row
      at[m] = row + (uint64_t)dt * stride32 + off;
    }
    u32x4 r[kGatherUnroll];
#pragma unroll
    for (int m = 0; m < kGatherUnroll; ++m) r[m] = *(const u32x4*)at[m];
#pragma unroll
    for (int m = 0; m < kGatherUnroll; ++m) __builtin_nontemporal_store(r[m], out + e0 + es[m]);
    // carry the pass's first vector forward by one pass
    const uint32_t x = r0 + kPass;
    const uint32_t du = small_div(x, vpu_m40);
    r0 = x - du * (uint32_t)vpu;
    const uint32_t hq = hd0 + du;
    const uint32_t dt = small_div(hq, h_m40);
    hd0 = hq - dt * h32;
    row += (uint64_t)dt * stride32;
  }
}

// Heads: workgroup w copies the 1024 vectors (16 KiB) of the send buffer
// from vector 1024 w on, or what of them the call fills.  Step descriptors
// are in step order with ascending first units (idle steps at their send
// offset), so the step holding the range's first unit is the last one
// starting at or before it: a search in which every thread tests one step
// per round (with at most 256 steps, one round whose loads go out together
// with the header's).  The workgroup then walks the steps its range meets.
// Every descriptor, its reciprocals included, is checked against the
// activations and the send buffer before its range is copied.
__global__ void __launch_bounds__(kGatherThreads) gather_heads_kernel(
    const unsigned char* __restrict__ src, const StepDesc* __restrict__ desc, const int32_t* __restrict__ u0s,
    const PackHeader* hdr, int32_t k_max, int64_t T, int64_t unit, int32_t vpu, uint64_t vpu_m40,
    uint64_t vpu_m64, int64_t cap_units, unsigned char* __restrict__ send, int32_t* status) {
  const int tid = threadIdx.x;
  const int64_t v0 = (int64_t)blockIdx.x * kGatherPass;
  const bool one_round = k_max <= kGatherThreads;
  const int32_t my_u0 = one_round && tid < k_max ? u0s[tid] : 0;
  const PackHeader hd = *hdr;
  const int K = hd.n_steps;
  if (*status != 0 || K <= 0) return;
  if (K > k_max) {   // a workspace not prepared for this k_max
    if (blockIdx.x == 0 && tid == 0) report(status, VP_ERR_INVALID_ARGUMENT);
    return;
  }
  if (hd.units < 0 || hd.units > cap_units) return;
  const int64_t nvec = hd.units * vpu;
  if (v0 >= nvec) return;
  const int64_t v1 = v0 + kGatherPass < nvec ? v0 + kGatherPass : nvec;
  const int64_t u_first = (int64_t)div64((uint64_t)v0, vpu_m64);
  const int64_t token_stride = hd.token_stride;
  // the last step whose first unit is at or before u_first (step 0 starts
  // at unit 0)
  int lo = 0;
  if (one_round) {
    const int c = __syncthreads_count(tid < K && my_u0 <= u_first);
    lo = c > 1 ? c - 1 : 0;
  } else {
    int hi = K;
    while (hi - lo > 1) {
      const int stride = (hi - lo + kGatherThreads - 1) / kGatherThreads;
      const int s = lo + tid * stride;
      const int c = __syncthreads_count(s < hi && u0s[s] <= u_first);
      lo += (c > 1 ? c - 1 : 0) * stride;
      hi = lo + stride < hi ? lo + stride : hi;
    }
  }
  for (int s = lo; s < K; ++s) {
    const StepDesc d = desc[s];
    const int64_t sv0 = (int64_t)d.u0 * vpu, sv1 = sv0 + (int64_t)d.nu * vpu;
    if (sv0 >= v1) break;
    const int64_t a = sv0 > v0 ? sv0 : v0, b = sv1 < v1 ? sv1 : v1;
    if (a >= b) continue;
    const uint64_t h = (uint64_t)d.h;
    if (d.h < 1 || d.h0 < 0 || ((int64_t)d.h0 + d.h) * unit > token_stride || d.u0 < 0 ||
        (int64_t)d.u0 + d.nu > cap_units || d.first < 0 || d.first + d.nu > T * d.h ||
        (d.h_m40 - 1) * h >= (uint64_t(1) << 40) || d.h_m40 * h < (uint64_t(1) << 40) ||
        (h == 1 ? d.h_m64 != 0 : d.h_m64 == 0 || __umul64hi(d.h_m64, h) == 0 || __umul64hi(d.h_m64 - 1, h) != 0)) {
      if (tid == 0) report(status, VP_ERR_INVALID_ARGUMENT);
      return;
    }
    copy_heads_range<kGatherThreads>(src, send, d, a, b, sv0, vpu, vpu_m40, vpu_m64, unit, token_stride, tid);
  }
}

struct FusedHeadsArgs {
  const unsigned char* src;
  unsigned char* send;
  int32_t N, self, k_max, vpu;
  int64_t unit, T, token_stride, send_capacity, heads_per_row;
  uint64_t vpu_m40, vpu_m64;
  const int32_t *Kp, *dst;
  const int64_t *bytes, *send_off, *stream_off, *head_lo;
  int64_t* step_off;
  PackHeader* hdr;   // the workspace is left as the two-kernel prepare leaves it
  StepDesc* desc;
  int32_t* u0s;
  int32_t* status;
};

// Heads with the planner's layout, at most 512 steps and 1024 ranks, in one
// kernel (prepare and copy): every workgroup checks the whole schedule
// itself, one step per thread, with the checks of the two-kernel prepare,
// before it copies anything -- all workgroups read the same schedule, so
// either every one copies or none does -- and keeps the descriptors in LDS;
// workgroup 0 writes step_off and the workspace.  The copy is the gather's,
// over ranges of two passes of 2048 vectors (64 KiB): fewer, larger
// workgroups than the gather's, since every workgroup repeats the schedule
// reads (measured best against one, four and eight passes).
constexpr int kFusedThreads = 512;
constexpr int kFusedPass = 2 * kFusedThreads * kGatherUnroll;   // vectors per workgroup

__global__ void __launch_bounds__(kFusedThreads) pack_heads_kernel(FusedHeadsArgs a) {
  __shared__ StepDesc sd[kFusedThreads];
  __shared__ int64_t hls[kHeadLoLds];
  __shared__ int64_t ends[kFusedThreads];   // where each step's slice ends
  const int tid = threadIdx.x;
  const size_t o = (size_t)tid * a.N + a.self;
  HeadsStep st{0, 0, 0, 0, 0};
  if (tid < a.k_max) {
    st.x = a.bytes[o];
    st.so = a.send_off[o];
    st.co = a.stream_off[o];
    st.j = a.dst[o];
  }
  for (int b = tid; b <= a.N; b += kFusedThreads) hls[b] = a.head_lo[b];
  const int K = *a.Kp, stat = *a.status;
  ends[tid] = st.so + st.x;
  const bool bad_k = K < 0 || K > a.k_max;
  const bool lead = blockIdx.x == 0;
  if (lead && tid == 0) {
    a.hdr->n_steps = bad_k ? 0 : K;
    a.hdr->token_stride = a.token_stride;
    if (bad_k) report(a.status, VP_ERR_INVALID_ARGUMENT);
    if (K == 0) {
      a.step_off[0] = 0;
      a.hdr->units = 0;
    }
  }
  __syncthreads();
  if (bad_k || stat != 0 || K == 0) return;
  st.prev_end = tid > 0 ? ends[tid - 1] : 0;
  StepDesc d;
  int err = 0;
  if (tid < K)
    err = heads_step_desc(
        st, [&](int b) { return hls[b]; }, a.N, a.self, a.unit, a.T, a.heads_per_row, a.send_capacity, d);
  if (__syncthreads_count(err != 0) != 0) {
    if (lead && err != 0) report(a.status, err);
    return;
  }
  if (tid < K) {
    sd[tid] = d;
    if (lead) {
      a.step_off[tid] = st.so;
      a.desc[tid] = d;
      a.u0s[tid] = d.u0;
      if (tid == K - 1) {
        a.step_off[K] = st.so + st.x;
        a.hdr->units = (st.so + st.x) / a.unit;
      }
    }
  }
  __syncthreads();
  const int64_t nvec = ((int64_t)sd[K - 1].u0 + sd[K - 1].nu) * a.vpu;
  const int64_t v0 = (int64_t)blockIdx.x * kFusedPass;
  if (v0 >= nvec) return;
  const int64_t v1 = v0 + kFusedPass < nvec ? v0 + kFusedPass : nvec;
  const int64_t u_first = (int64_t)div64((uint64_t)v0, a.vpu_m64);
  const int c = __syncthreads_count(tid < K && d.u0 <= u_first);
  for (int s = c > 1 ? c - 1 : 0; s < K; ++s) {
    const StepDesc ds = sd[s];
    const int64_t sv0 = (int64_t)ds.u0 * a.vpu, sv1 = sv0 + (int64_t)ds.nu * a.vpu;
    if (sv0 >= v1) break;
    const int64_t lo = sv0 > v0 ? sv0 : v0, hi = sv1 < v1 ? sv1 : v1;
    if (lo < hi)
      copy_heads_range<kFusedThreads>(a.src, a.send, ds, lo, hi, sv0, a.vpu, a.vpu_m40, a.vpu_m64, a.unit,
                                      a.token_stride, tid);
  }
}

size_t desc_bytes(int32_t k_max) {
  return align_up((size_t)k_max * sizeof(StepDesc) + 16, 256) + align_up((size_t)k_max * 4, 256);
}

constexpr size_t kHeader = 256;   // room for the PackHeader

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
  PackHeader* hdr = (PackHeader*)ws;
  StepDesc* desc = (StepDesc*)(ws + kHeader);
  int32_t* n_desc = (int32_t*)(ws + kHeader + (size_t)a.k_max * sizeof(StepDesc));
  int32_t* u0s = (int32_t*)(ws + kHeader + align_up((size_t)a.k_max * sizeof(StepDesc) + 16, 256));
  char* rest = ws + kHeader + desc_bytes(a.k_max);
  unsigned long long* lst = (unsigned long long*)rest;
  // heads: a unit's vectors and a destination's heads are divisors of the
  // gather's 32-bit divisions
  if (a.mode == 1) {
    if (a.token_stride / a.unit > ((int64_t)1 << 15))
      return set_error(VP_ERR_UNSUPPORTED, "more than 2^15 heads per token");
    if (a.unit >= ((int64_t)1 << 23)) return set_error(VP_ERR_UNSUPPORTED, "head units of 8 MiB or more");
    if (a.token_stride >= ((int64_t)1 << 32)) return set_error(VP_ERR_UNSUPPORTED, "token rows of 4 GiB or more");
    if (a.send_capacity >= ((int64_t)1 << 52)) return set_error(VP_ERR_UNSUPPORTED, "send buffer too large");
    // the gather's 64-bit divisions: send vectors by a unit's vectors, stream
    // positions (below T * heads) by a destination's heads
    const unsigned __int128 vpu128 = (unsigned __int128)(a.unit / 16), hmax = (unsigned __int128)(a.token_stride / a.unit);
    if ((unsigned __int128)(a.send_capacity / 16) * vpu128 >= ((unsigned __int128)1 << 63) ||
        (unsigned __int128)a.T * hmax * hmax >= ((unsigned __int128)1 << 63))
      return set_error(VP_ERR_UNSUPPORTED, "too many heads or head units for the gather's divisions");
  }

  // heads with the planner's layout and a short schedule: prepare and copy
  // in one kernel (one workgroup per 64 KiB of send capacity, at least one)
  if (a.mode == 1 && layout && a.stages == 3 && a.k_max <= kFusedThreads && a.N + 1 <= kHeadLoLds) {
    const int64_t vpu = a.unit / 16;
    const int64_t blocks = std::max<int64_t>(1, (a.send_capacity / 16 + kFusedPass - 1) / kFusedPass);
    if (blocks >= ((int64_t)1 << 31)) return set_error(VP_ERR_UNSUPPORTED, "send buffer too large");
    FusedHeadsArgs fa{(const unsigned char*)a.src, (unsigned char*)a.send, a.N, a.self_rank, a.k_max, (int32_t)vpu,
                      a.unit, a.T, a.token_stride, a.send_capacity, a.token_stride / a.unit,
                      magic40((uint64_t)vpu), magic64((uint64_t)vpu),
                      a.K, a.dst, a.bytes, a.send_off, a.stream_off, a.head_lo, a.step_off, hdr, desc, u0s,
                      a.status};
    hipLaunchKernelGGL(pack_heads_kernel, dim3((unsigned)blocks), dim3(kFusedThreads), 0, s, fa);
    if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "pack launch failed");
    return VP_OK;
  }

  if (a.stages & 1) {
    uint32_t gen = ++g_generation;
    if (gen == 0) gen = ++g_generation;   // zero is the value of a cleared workspace
    IndexArgs ia{a.mode, a.k, a.self_rank, a.N, a.k_max, a.unit, a.T, a.token_stride, a.send_capacity,
                 a.token_stride / a.unit, gen,
                 a.sorted_tok, a.sorted_slot, desc, u0s, n_desc, a.K, a.dst, a.bytes, a.send_off, a.stream_off,
                 a.mode == 0 ? a.dest_off : a.head_lo, a.step_off, hdr, lst, a.status};
    if (!layout) {
      SliceArgs sa{a.mode, a.K, a.dst, a.bytes, a.k_max, a.N, a.self_rank, a.unit, a.T, a.send_capacity,
                   a.token_stride, a.mode == 0 ? a.dest_off : a.head_lo, a.step_off, desc, u0s, n_desc, hdr,
                   a.status};
      if (hipFuncSetAttribute((const void*)slices_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                              (int)lds) != hipSuccess)
        return set_error(VP_ERR_HIP, "cannot raise the slice kernel's LDS limit");
      hipLaunchKernelGGL(slices_kernel, dim3(1), dim3(1024), lds, s, sa);
    } else if (a.mode == 1) {
      const unsigned blocks = (unsigned)std::max<int64_t>(1, (a.k_max + kIndexThreads - 1) / kIndexThreads);
      hipLaunchKernelGGL(heads_index_kernel, dim3(blocks), dim3(kIndexThreads), 0, s, ia);
    }
    if (a.mode == 0) {
      // a step holds up to one destination's whole stream: split it over up
      // to 16 workgroups so that a thread handles about two of its units
      const int64_t units = a.T * a.k;
      const int64_t per_step = (units + a.N - 1) / std::max(1, a.N);
      const int ny = (int)std::min<int64_t>(16, std::max<int64_t>(1, (per_step + 2 * kIndexThreads - 1) /
                                                                        (2 * kIndexThreads)));
      hipLaunchKernelGGL(index_kernel, dim3(a.k_max, ny), dim3(kIndexThreads), 0, s, ia);
    }
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
    // one workgroup per 16 KiB of send capacity
    const int64_t blocks = (a.send_capacity / 16 + kGatherPass - 1) / kGatherPass;
    if (blocks >= ((int64_t)1 << 31)) return set_error(VP_ERR_UNSUPPORTED, "send buffer too large");
    if (blocks > 0)
      hipLaunchKernelGGL(gather_heads_kernel, dim3((unsigned)blocks), dim3(kGatherThreads), 0, s,
                         (const unsigned char*)a.src, desc, u0s, hdr, a.k_max, a.T, a.unit, (int32_t)vpu,
                         magic40((uint64_t)vpu), magic64((uint64_t)vpu), a.send_capacity / a.unit,
                         (unsigned char*)a.send, a.status);
  }
  if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "pack launch failed");
  return VP_OK;
}

}  // namespace vp
