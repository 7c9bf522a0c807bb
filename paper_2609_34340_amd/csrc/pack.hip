// vp_pack: channel-ordered send buffers (Sec. 5 "Device-resident buffer
// layout").  For the steps in which this rank's lane carries bytes, in
// schedule order, the next x bytes of the stream to that step's destination
// are appended to the send buffer.
//
// Kernels
//   slices   one block; after one round of global loads everything runs in
//            LDS: step offsets (exclusive scan of this rank's lane volumes)
//            and each step's offset inside its destination's stream (a
//            stable counting sort of the steps by destination -- per-wave
//            ballot ranks over contiguous chunks, one scan over destinations
//            and waves -- then a scan of the volumes in (destination, step)
//            order).  For token rows it also clears the per-token copy
//            counters.
//   index    one wavefront per step.  Rows: every packed unit is one copy of
//            a token row, and its send-unit index joins that token's copy
//            list.  Heads: the source byte offset of every packed unit.
//   scatter  rows: one workgroup per token reads the row once into registers
//            and stores it to each of its copies, so a source row leaves HBM
//            once however many destinations it has.
//   gather   heads: grid-stride 16-byte copy of the units (each is read
//            once) with non-temporal stores.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "internal.h"

namespace vp {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ inline void report(int32_t* status, int code) { atomicCAS(status, 0, code); }

__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Exclusive block scan of v over 1024 threads; returns the exclusive prefix
// and writes the block total to *total.
__device__ int64_t block_excl_scan(int64_t v, int64_t* wsum, int64_t* total) {
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int64_t s = v;
  for (int o = 1; o < 64; o <<= 1) {
    int64_t y = __shfl_up(s, o);
    if (lane >= o) s += y;
  }
  if (lane == 63) wsum[w] = s;
  __syncthreads();
  int64_t before = 0, all = 0;
  for (int k = 0; k < 16; ++k) {
    if (k < w) before += wsum[k];
    all += wsum[k];
  }
  __syncthreads();
  *total = all;
  return before + s - v;
}

struct SliceArgs {
  int mode;
  const int32_t *Kp, *dst;
  const int64_t* bytes;
  int32_t k_max, N, self;
  int64_t unit, T, send_capacity, token_stride;
  const int64_t* dest_off;   // rows
  const int64_t* head_lo;    // heads
  int64_t* step_off;
  int64_t* cstream;          // per step: offset inside the destination stream (bytes)
  int32_t* tcnt;             // rows: per-token copy counters, cleared here
  int32_t* status;
};

// Dynamic LDS of the slice kernel for schedule capacity k_max and N ranks.
size_t slice_lds_bytes(int32_t k_max, int32_t N) {
  const size_t rw = std::max<size_t>((size_t)k_max, (size_t)8 * N);
  return (size_t)k_max * (8 + 4 + 4) + rw * 8 + (size_t)N * (8 + 4);
}

__global__ void __launch_bounds__(1024) slices_kernel(SliceArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int N = a.N;
  const int RW = a.k_max > 8 * N ? a.k_max : 8 * N;
  int64_t* xk = (int64_t*)smem;          // k_max: this rank's lane volume of step k (0: idle or rejected)
  int64_t* xs = xk + a.k_max;            // RW: volumes in (destination, step) order, then their scan
  int32_t* wcnt = (int32_t*)xs;          // [16][N]: per-wave destination counts (ranking only)
  int64_t* len = xs + RW;                // N: stream length of each destination (bytes)
  int32_t* jv = (int32_t*)(len + N);     // k_max: destination of step k, N when idle
  int32_t* pos = jv + a.k_max;           // k_max: position in (destination, step) order
  int32_t* run = pos + a.k_max;          // N: first position of each destination
  __shared__ int64_t wsum[16];
  __shared__ int64_t carry;
  __shared__ int32_t Ks;

  if (tid == 0) {
    int K = *a.Kp;
    if (K < 0 || K > a.k_max) {
      report(a.status, VP_ERR_INVALID_ARGUMENT);
      K = 0;
    }
    // every head a destination owns must lie inside the token row
    if (a.mode == 1 && (a.head_lo[0] < 0 || a.head_lo[N] * a.unit > a.token_stride)) {
      report(a.status, VP_ERR_INVALID_ARGUMENT);
      K = 0;
    }
    Ks = K;
    carry = 0;
  }
  for (int i = tid; i < 16 * N; i += 1024) wcnt[i] = 0;
  if (a.mode == 0)
    for (int64_t t = tid; t < a.T; t += 1024) a.tcnt[t] = 0;
  __syncthreads();
  const int K = Ks;

  // 1. the only global loads: lane volumes and destinations, stream lengths
  for (int k = tid; k < K; k += 1024) {
    int64_t x = a.bytes[(size_t)k * N + a.self];
    const int j = a.dst[(size_t)k * N + a.self];
    int b = N;
    if (x != 0) {
      if (x < 0 || x % a.unit != 0 || j < 0 || j >= N || j == a.self) {
        report(a.status, VP_ERR_INVALID_ARGUMENT);
        x = 0;
      } else {
        b = j;
      }
    }
    xk[k] = x;
    jv[k] = b;
  }
  for (int b = tid; b < N; b += 1024)
    len[b] = a.mode == 0 ? (a.dest_off[b + 1] - a.dest_off[b]) * a.unit
                         : a.T * (a.head_lo[b + 1] - a.head_lo[b]) * a.unit;
  __syncthreads();

  // 2. step offsets: exclusive scan of the lane volumes in schedule order
  for (int k0 = 0; k0 < K; k0 += 1024) {
    const int k = k0 + tid;
    const int64_t x = k < K ? xk[k] : 0;
    int64_t tot;
    const int64_t e = block_excl_scan(x, wsum, &tot);
    if (k < K) a.step_off[k] = carry + e;
    __syncthreads();
    if (tid == 0) carry += tot;
    __syncthreads();
  }
  if (tid == 0) {
    a.step_off[K] = carry;
    if (carry > a.send_capacity) report(a.status, VP_ERR_CAPACITY);
    carry = 0;
  }

  // 3. stable rank of every carrying step among the steps to its
  //    destination: wave v ranks the chunk [v*C, (v+1)*C) with ballot match
  //    masks, then destinations and waves are scanned in (destination, wave)
  //    order.
  const int C = (((K + 15) / 16) + 63) & ~63;
  {
    int bits = 0;
    while ((1 << bits) < N) ++bits;
    const uint64_t lt = lane == 0 ? 0ull : (~0ull >> (64 - lane));
    int32_t* mine = wcnt + w * N;
    const int k_lo = w * C, k_hi = k_lo + C < K ? k_lo + C : K;
    for (int k0 = k_lo; k0 < k_hi; k0 += 64) {
      const int k = k0 + lane;
      const int b = k < k_hi ? jv[k] : N;
      const bool live = b < N;
      uint64_t same = __ballot(live);
      for (int bt = 0; bt < bits; ++bt) {
        const uint64_t ones = __ballot(live && ((b >> bt) & 1));
        same &= ((b >> bt) & 1) ? ones : ~ones;
      }
      int r = 0;
      if (live) r = mine[b] + __popcll(same & lt);
      wave_sync();
      if (live && (same & lt) == 0) mine[b] += __popcll(same);
      wave_sync();
      if (live) pos[k] = r;
    }
  }
  __syncthreads();
  for (int b0 = 0; b0 < N; b0 += 1024) {
    const int b = b0 + tid;
    int64_t tb = 0;
    if (b < N)
      for (int v = 0; v < 16; ++v) tb += wcnt[v * N + b];
    int64_t tot;
    const int64_t e = block_excl_scan(tb, wsum, &tot);
    if (b < N) {
      int acc = (int)(carry + e);
      run[b] = acc;
      for (int v = 0; v < 16; ++v) {
        const int c = wcnt[v * N + b];
        wcnt[v * N + b] = acc;
        acc += c;
      }
    }
    __syncthreads();
    if (tid == 0) carry += tot;
    __syncthreads();
  }
  const int KL = (int)carry;  // carrying steps
  for (int k = tid; k < K; k += 1024)
    if (jv[k] < N) pos[k] += wcnt[(k / C) * N + jv[k]];
  __syncthreads();

  // 4. volumes in (destination, step) order, then one exclusive scan
  for (int k = tid; k < K; k += 1024)
    if (jv[k] < N) xs[pos[k]] = xk[k];
  if (tid == 0) carry = 0;
  __syncthreads();
  for (int k0 = 0; k0 < KL; k0 += 1024) {
    const int k = k0 + tid;
    const int64_t x = k < KL ? xs[k] : 0;
    int64_t tot;
    const int64_t e = block_excl_scan(x, wsum, &tot);
    if (k < KL) xs[k] = carry + e;
    __syncthreads();
    if (tid == 0) carry += tot;
    __syncthreads();
  }

  // 5. offset of each step inside its destination's stream; bounds check
  for (int k = tid; k < K; k += 1024) {
    const int b = jv[k];
    if (b == N) {
      a.cstream[k] = 0;
      continue;
    }
    const int64_t c = xs[pos[k]] - xs[run[b]];
    if (c + xk[k] > len[b]) report(a.status, VP_ERR_INVALID_ARGUMENT);
    a.cstream[k] = c;
  }
}

struct IndexArgs {
  int mode;
  const int32_t *Kp, *dst;
  const int64_t* bytes;
  int32_t N, self, k;
  int64_t unit, T, token_stride;
  const int32_t* sorted_tok;
  const int64_t* dest_off;
  const int64_t* head_lo;
  const int64_t* step_off;
  const int64_t* cstream;
  int32_t* tcnt;             // rows: copies recorded per token
  int32_t* lst;              // rows: [T][k] send-unit index of each copy
  int64_t* src_off;          // heads: source byte offset per send unit
  int32_t* status;
};

__global__ void __launch_bounds__(64) index_kernel(IndexArgs a) {
  const int k = blockIdx.x, lane = threadIdx.x;
  if (k >= *a.Kp || *a.status != 0) return;
  const int64_t x = a.bytes[(size_t)k * a.N + a.self];
  if (x <= 0) return;
  const int j = a.dst[(size_t)k * a.N + a.self];
  const int64_t nu = x / a.unit, u0 = a.step_off[k] / a.unit, p0 = a.cstream[k] / a.unit;
  if (a.mode == 0) {
    const int64_t first = a.dest_off[j] + p0;
    for (int64_t u = lane; u < nu; u += 64) {
      const int64_t tok = a.sorted_tok[first + u];
      if (tok < 0 || tok >= a.T) {
        report(a.status, VP_ERR_INVALID_ARGUMENT);
        continue;
      }
      const int slot = atomicAdd(&a.tcnt[tok], 1);
      if (slot >= a.k) {
        report(a.status, VP_ERR_INVALID_ARGUMENT);
        continue;
      }
      a.lst[tok * a.k + slot] = (int32_t)(u0 + u);
    }
  } else {
    const int64_t h0 = a.head_lo[j], h = a.head_lo[j + 1] - h0;
    for (int64_t u = lane; u < nu; u += 64) {
      const int64_t p = p0 + u, tok = p / h, hd = h0 + (p - tok * h);
      a.src_off[u0 + u] = tok * a.token_stride + hd * a.unit;
    }
  }
}

constexpr int kScatterThreads = 256;
constexpr int kScatterUnroll = 4;

// Rows: workgroup per token (grid-stride); the row is loaded once and
// stored to every send unit on the token's copy list.
__global__ void __launch_bounds__(kScatterThreads) scatter_rows_kernel(
    const unsigned char* __restrict__ src, const int32_t* __restrict__ tcnt, const int32_t* __restrict__ lst,
    int64_t T, int k, int64_t unit, int64_t vpu, unsigned char* __restrict__ send, const int32_t* status) {
  if (*status != 0) return;
  const int tid = threadIdx.x;
  for (int64_t t = blockIdx.x; t < T; t += gridDim.x) {
    int n = tcnt[t];
    n = n < k ? n : k;
    if (n <= 0) continue;
    const u32x4* row = (const u32x4*)(src + t * unit);
    const int32_t* copies = lst + t * k;
    for (int64_t i0 = tid; i0 < vpu; i0 += kScatterThreads * kScatterUnroll) {
      u32x4 r[kScatterUnroll];
#pragma unroll
      for (int m = 0; m < kScatterUnroll; ++m) {
        const int64_t i = i0 + m * kScatterThreads;
        if (i < vpu) r[m] = row[i];
      }
      for (int c = 0; c < n; ++c) {
        u32x4* d = (u32x4*)(send + (int64_t)copies[c] * unit);
#pragma unroll
        for (int m = 0; m < kScatterUnroll; ++m) {
          const int64_t i = i0 + m * kScatterThreads;
          if (i < vpu) __builtin_nontemporal_store(r[m], d + i);
        }
      }
    }
  }
}

constexpr int kGatherThreads = 256;
constexpr int kGatherUnroll = 4;

// Heads: grid-stride over the 16-byte vectors of the send buffer.
__global__ void __launch_bounds__(kGatherThreads) gather_kernel(const unsigned char* __restrict__ src,
                                                                const int64_t* __restrict__ src_off,
                                                                const int32_t* Kp, const int64_t* step_off,
                                                                int64_t unit, int64_t vpu, uint64_t magic,
                                                                unsigned char* __restrict__ send,
                                                                const int32_t* status) {
  if (*status != 0) return;
  const int64_t total_vec = step_off[*Kp] / 16;
  const int64_t stride = (int64_t)gridDim.x * kGatherThreads;
  int64_t v = (int64_t)blockIdx.x * kGatherThreads + threadIdx.x;
  for (; v + (kGatherUnroll - 1) * stride < total_vec; v += kGatherUnroll * stride) {
    u32x4 r[kGatherUnroll];
#pragma unroll
    for (int m = 0; m < kGatherUnroll; ++m) {
      const uint64_t vv = (uint64_t)(v + m * stride);
      const int64_t u = (int64_t)__umul64hi(vv << 16, magic);
      const int64_t in = (int64_t)vv - u * vpu;
      r[m] = *(const u32x4*)(src + src_off[u] + in * 16);
    }
#pragma unroll
    for (int m = 0; m < kGatherUnroll; ++m)
      __builtin_nontemporal_store(r[m], (u32x4*)(send + (v + m * stride) * 16));
  }
  for (; v < total_vec; v += stride) {
    const int64_t u = (int64_t)__umul64hi((uint64_t)v << 16, magic);
    const int64_t in = v - u * vpu;
    u32x4 r = *(const u32x4*)(src + src_off[u] + in * 16);
    __builtin_nontemporal_store(r, (u32x4*)(send + v * 16));
  }
}
size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

}  // namespace

size_t pack_workspace(int32_t k_max, int64_t send_capacity, int64_t unit, int64_t T, int32_t k) {
  const size_t head = align_up((size_t)(k_max + 1) * sizeof(int64_t), 256);
  if (k > 0) return head + align_up((size_t)T * sizeof(int32_t), 256) + (size_t)T * (size_t)k * sizeof(int32_t);
  return head + ((size_t)(send_capacity / unit) + 1) * sizeof(int64_t);
}

vp_status launch_pack(const PackLaunch& a, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  const size_t lds = slice_lds_bytes(a.k_max, a.N);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return set_error(VP_ERR_HIP, "hipGetDevice failed");
  int lds_max = 0;
  if (hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
    return set_error(VP_ERR_HIP, "hipDeviceGetAttribute failed");
  if (lds + 1024 > (size_t)lds_max) return set_error(VP_ERR_UNSUPPORTED, "k_max too large for the slice table");
  if (a.unit % 16 != 0) return set_error(VP_ERR_INVALID_ARGUMENT, "unit must be a multiple of 16");
  if ((a.mode == 0) != (a.k > 0)) return set_error(VP_ERR_INVALID_ARGUMENT, "top-k must be > 0 exactly for rows");
  // rows record send-unit indices as int32
  if (a.mode == 0 && a.send_capacity / a.unit >= ((int64_t)1 << 31))
    return set_error(VP_ERR_UNSUPPORTED, "send buffer too large");
  char* ws = (char*)a.ws;
  int64_t* cstream = (int64_t*)ws;
  char* rest = ws + align_up((size_t)(a.k_max + 1) * sizeof(int64_t), 256);
  int32_t* tcnt = (int32_t*)rest;
  int32_t* lst = (int32_t*)(rest + align_up((size_t)a.T * sizeof(int32_t), 256));
  int64_t* src_off = (int64_t*)rest;

  if (a.stages & 1) {
    SliceArgs sa{a.mode, a.K, a.dst, a.bytes, a.k_max, a.N, a.self_rank, a.unit, a.T, a.send_capacity,
                 a.token_stride, a.dest_off, a.head_lo, a.step_off, cstream, tcnt, a.status};
    if (hipFuncSetAttribute((const void*)slices_kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
        hipSuccess)
      return set_error(VP_ERR_HIP, "cannot raise the slice kernel's LDS limit");
    hipLaunchKernelGGL(slices_kernel, dim3(1), dim3(1024), lds, s, sa);

    IndexArgs ia{a.mode, a.K, a.dst, a.bytes, a.N, a.self_rank, a.k, a.unit, a.T, a.token_stride, a.sorted_tok,
                 a.dest_off, a.head_lo, a.step_off, cstream, tcnt, lst, src_off, a.status};
    hipLaunchKernelGGL(index_kernel, dim3(a.k_max), dim3(64), 0, s, ia);
  }
  if (!(a.stages & 2)) {
    if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "pack launch failed");
    return VP_OK;
  }
  const int64_t vpu = a.unit / 16;
  if (a.mode == 0) {
    if (a.T > 0) {
      const int64_t blocks = std::min<int64_t>(a.T, 16384);
      hipLaunchKernelGGL(scatter_rows_kernel, dim3((unsigned)blocks), dim3(kScatterThreads), 0, s,
                         (const unsigned char*)a.src, tcnt, lst, a.T, a.k, a.unit, vpu, (unsigned char*)a.send,
                         a.status);
    }
  } else {
    // u = floor(v / vpu) = mulhi(v << 16, ceil(2^48 / vpu)) for v < 2^48 / vpu
    const unsigned __int128 two48 = (unsigned __int128)1 << 48;
    const uint64_t magic = (uint64_t)((two48 + (unsigned __int128)vpu - 1) / (unsigned __int128)vpu);
    const int64_t max_vec = a.send_capacity / 16;
    if (max_vec >= ((int64_t)1 << 48) / vpu) return set_error(VP_ERR_UNSUPPORTED, "send buffer too large");
    int64_t blocks = (max_vec + kGatherThreads * kGatherUnroll - 1) / (kGatherThreads * kGatherUnroll);
    blocks = std::max<int64_t>(1, std::min<int64_t>(blocks, 8192));
    hipLaunchKernelGGL(gather_kernel, dim3((unsigned)blocks), dim3(kGatherThreads), 0, s,
                       (const unsigned char*)a.src, src_off, a.K, a.step_off, a.unit, vpu, magic,
                       (unsigned char*)a.send, a.status);
  }
  if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "pack launch failed");
  return VP_OK;
}

}  // namespace vp
