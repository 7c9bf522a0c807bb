// vp_plan: online channel-guided demand decomposition (Sec. 4.2, Alg. 2) as
// one persistent workgroup of 1024 threads that runs the whole iteration
// loop on the device (vp_plan_batch: one such workgroup per matrix).
//
// Per iteration:
//   1. shape scores, Eq. (5)-(6), from node-block aggregates kept in LDS:
//      A = sum over nodes of the diagonal node block of D-hat and B_k = sum of
//      the blocks (n, n+k).  A shape (k, L, R) scores sum A.L + sum B_k.R,
//      which equals sum D-hat.M.  The aggregates are kept in units of the
//      pack granule as int32 (every demand entry is a whole number of units,
//      so scores keep their order).  The B part depends on a pattern only
//      through its set of NIC lanes: a few lanes per distinct set find the
//      set's best shift while other threads compute every pattern's A part;
//      one thread per pattern then adds the two and the block takes the
//      argmax of packed 64-bit keys (ties to the lowest canonical shape);
//   2. for the families of the best shape: the cluster-level out/in lists of
//      every group and the binding credits h' = min(D^rem_ij, cap) (Eq. (7)
//      scaled by tau) of every instance and endpoint pair, into LDS, with
//      the shuffled starts' permutations drawn on the idle wavefronts;
//   3. MultiStartAA (Eq. (8)): one wavefront per (family, start).  Each lane
//      owns up to a few groups for both AA halves and keeps their source and
//      destination assignments and credit rows in registers, so a half-step
//      is one LDS round trip (read the other side, write back);
//   4. Evaluate (Eq. (9)-(10)), the exact utility argmax in 128-bit, by each
//      wavefront that writes the winner (a one-family shape needs only its
//      best start);
//   5. the activation is appended and D^rem (global memory, touched by this
//      one workgroup only) is updated; the per-rank stream offsets are
//      completed by stream_off_kernel after the loop.
// No host round trip happens between iterations.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <string>

#include "internal.h"

namespace vp {
namespace {

constexpr int kWaves = kPlanThreads / 64;
constexpr int kMaxQG = kMaxSlotsPerNode * kMaxGpusPerSwitch;   // lanes per node
constexpr int kMaxLTerms = 3 * kMaxSlotsPerNode;   // PIX, PXB and NIC entries of one diagonal block
constexpr uint32_t kRawSaturated = 0xFFFFFFFEu;     // residual too large for 32 bits: reload it

// Phase timing, compiled only with -DVP_PHASE_STAMPS (phase_stamps.py builds
// such a copy): thread 0 of workgroup 0 stores the cycle counter at each
// phase boundary of every iteration, row = iteration (4096 rows of 16):
// columns 0-8 open the phases, 9-14 mark points inside them (thread 0's
// gather items done, the start draws done, the best start read, the
// update's reads done, its stores issued, the shared totals written).
#ifdef VP_PHASE_STAMPS
__device__ unsigned long long g_phase_stamps[4096 * 16];
#define VP_STAMP(k)                                                                                  \
  do {                                                                                               \
    if (threadIdx.x == 0 && blockIdx.x == 0)                                                         \
      g_phase_stamps[(stamp_it < 4095 ? stamp_it : 4095) * 16 + (k)] = __builtin_readcyclecounter(); \
  } while (0)
#else
#define VP_STAMP(k) ((void)0)
#endif

struct PairRes {
  int64_t F;
  // largest lane volume on a PCIe-rate path (PIX, PXB, SYS) and on a NIC
  // path: Eq. (10) needs only the largest volume / rate, and the classes of
  // one rate share a maximum
  int64_t xmax[2];
};

struct Shared {
  uint64_t key;
  int64_t total_rem, Lmax, tau, total_units;
  int64_t cap[4];
  int32_t capu[4];
  int32_t K, err;
  int32_t huge;   // some demand entry reaches 2^42 bytes
};

struct PlanArgs {
  const int32_t* cat;
  DevCatalogLayout L;
  const int64_t* D;
  int64_t* Drem;
  int64_t k_target, lambda, unit;
  uint64_t seed;
  uint64_t odd_inv, odd_lim;
  int32_t unit_shift;
  int32_t n_start, i_aa, k_max, FC;
  int32_t LPS, SPT;   // shift scoring: lanes per NIC-lane set (a power of two) and shifts per lane
  int32_t LPS_log2;
  uint32_t qg_magic;  // ceil(2^32 / (Q g)): t / (Q g) = umulhi(t, qg_magic) for t < 2^16
  int32_t MLT, MRT;   // most diagonal-block terms of a pattern; largest NIC-lane set
  int32_t *K, *family, *dst, *inst;
  int64_t *bytes, *tau;
  int64_t *send_off, *stream_off;   // optional [k_max][N] buffer layout per rank
  int32_t* recv_src;                // optional [k_max][N]: the rank whose lane lands at each rank
  int32_t* status;
  int32_t batch;                    // matrices, one workgroup each; every buffer above holds `batch` of them
  // LDS layout (byte offsets)
  int32_t o_agg, o_terms, o_pfb, o_finfo;
  int32_t o_pair, o_outT, o_inT, o_ipos, o_ocls, o_iid, o_hp, o_raw, o_sl, o_dl, o_top;
  int32_t o_rset, o_psid, o_rbest, o_pbase, o_rp;
};

// Per-rank arrays of plan_kernel<g, MG> sit at compile-time offsets from the
// start of the dynamic LDS, sized for the most ranks the instantiation
// takes (64 MG groups of g): they are addressed with immediate offsets and
// hold no scalar register.  Everything else follows at host-computed offsets.
struct FixedLds {
  size_t rinfo, lastj, lastv, sacc, bx, brw, bsl, bdl, bid, end;
};
__host__ __device__ constexpr size_t a16(size_t x) { return (x + 15) / 16 * 16; }
__host__ __device__ constexpr FixedLds fixed_lds(size_t n) {
  FixedLds f{};
  f.rinfo = a16(sizeof(Shared));
  f.lastj = f.rinfo + 4 * n;
  f.lastv = a16(f.lastj + 4 * n);
  f.sacc = f.lastv + 8 * n;
  f.bx = f.sacc + 8 * n;
  f.brw = f.bx + 4 * n;
  f.bsl = f.brw + 4 * n;
  f.bdl = f.bsl + n;
  f.bid = f.bdl + n;
  f.end = a16(f.bid + n);
  return f;
}

// ------------------------------------------------------------------ helpers

__device__ inline void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Whole-wavefront reductions of the device library (DPP based); every lane
// receives the result.
extern "C" __device__ __attribute__((const)) long long __ockl_wfred_add_i64(long long);
extern "C" __device__ __attribute__((const)) long long __ockl_wfred_max_i64(long long);
extern "C" __device__ __attribute__((const)) unsigned long long __ockl_wfred_max_u64(unsigned long long);
__device__ inline int64_t wave_sum(int64_t v) { return __ockl_wfred_add_i64(v); }
__device__ inline int64_t wave_max(int64_t v) { return __ockl_wfred_max_i64(v); }
extern "C" __device__ __attribute__((const)) int __ockl_wfred_max_i32(int);
__device__ inline uint64_t wave_max_u(uint64_t v) { return __ockl_wfred_max_u64(v); }
__device__ inline int32_t wave_max32(int32_t v) { return __ockl_wfred_max_i32(v); }
// lane 0's value in every lane (the whole wavefront active)
__device__ inline int32_t lane0(int32_t v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ inline int64_t lane0(int64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)v);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int32_t)(v >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Binding credits are held in pack units as int32 (every credit is a whole
// number of units, so dividing by the unit keeps every comparison).  A self
// pair holds kForbiddenU = -2^29: valid credits are below 2^27, so a sum of at
// most four credits that includes a self pair is negative (it loses to every
// assignment without one), and four self pairs still fit in 32 bits.
constexpr int32_t kForbiddenU = -(1 << 29);

// SplitMix64 (Steele, Lea, Flood 2014): key absorbs the fields one at a time.
constexpr uint64_t kGolden = 0x9E3779B97F4A7C15ull;
__device__ inline uint64_t sm_mix(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Utility order of Eq. (10): (S1, x1/b1) beats (S2, x2/b2) exactly.
__device__ inline bool utility_greater(int64_t S1, int64_t x1, int64_t b1, int64_t S2, int64_t x2,
                                       int64_t b2, int64_t lam) {
  if (S1 == 0) return false;
  if (S2 == 0) return true;
  typedef unsigned __int128 u128;
  u128 lhs = (u128)S1 * (u128)b1 * ((u128)lam * (u128)b2 + (u128)x2);
  u128 rhs = (u128)S2 * (u128)b2 * ((u128)lam * (u128)b1 + (u128)x1);
  return lhs > rhs;
}

// Lexicographic permutations of g elements.
template <int g>
struct Perms;
template <>
struct Perms<2> {
  static constexpr int n = 2;
  __device__ static int at(int p, int m) { return p ? 1 - m : m; }
};
template <>
struct Perms<3> {
  static constexpr int n = 6;
  __device__ static int at(int p, int m) {
    constexpr unsigned char t[6][3] = {{0, 1, 2}, {0, 2, 1}, {1, 0, 2}, {1, 2, 0}, {2, 0, 1}, {2, 1, 0}};
    return t[p][m];
  }
};
template <>
struct Perms<4> {
  static constexpr int n = 24;
  __device__ static int at(int p, int m) {
    constexpr unsigned char t[24][4] = {
        {0, 1, 2, 3}, {0, 1, 3, 2}, {0, 2, 1, 3}, {0, 2, 3, 1}, {0, 3, 1, 2}, {0, 3, 2, 1},
        {1, 0, 2, 3}, {1, 0, 3, 2}, {1, 2, 0, 3}, {1, 2, 3, 0}, {1, 3, 0, 2}, {1, 3, 2, 0},
        {2, 0, 1, 3}, {2, 0, 3, 1}, {2, 1, 0, 3}, {2, 1, 3, 0}, {2, 3, 0, 1}, {2, 3, 1, 0},
        {3, 0, 1, 2}, {3, 0, 2, 1}, {3, 1, 0, 2}, {3, 1, 2, 0}, {3, 2, 0, 1}, {3, 2, 1, 0}};
    return t[p][m];
  }
};

// Local family descriptor (16 bits): cls | src_slot<<2 | dst_slot<<5 |
// out_pos<<8 | rank_same<<10 | n_other<<12.  rank_same is the instance's rank
// among the in-instances of its destination slot of the same kind (same-node
// or cross-node lane), n_other the number of the other kind: cross-node
// in-instances precede same-node ones exactly when their source node is the
// lower one.
__device__ inline int d_cls(uint32_t w) { return w & 3; }
__device__ inline int d_ss(uint32_t w) { return (w >> 2) & 7; }
__device__ inline int d_ds(uint32_t w) { return (w >> 5) & 7; }
__device__ inline int d_opos(uint32_t w) { return (w >> 8) & 3; }
__device__ inline int d_rsame(uint32_t w) { return (w >> 10) & 3; }
__device__ inline int d_nother(uint32_t w) { return (w >> 12) & 7; }

// Per-family working set of the current chunk.
struct FamCtx {
  const uint16_t* outT;   // [G*g] out-instance t of (group, m)
  const uint16_t* inT;    // [G*g] in-instance t of (group, m)
  const int8_t* ipos;     // [G*g] position of the out-instance in its group's in-list if intra, else -1
  const uint8_t* ocls;    // [G*g] path class of the out-instance
  const int32_t* H;       // [N*g*g] credits (units; kForbiddenU for a self pair)
  int f;                  // global family index
};

// One (family, start) pair; executed by one whole wavefront.  `top` is the
// family's highest-credit triple packed as credit << 24 | (2^24 - 1 - (t*g*g +
// i*g + j)) (0 when no credit is positive); `rperm` holds, for a shuffled
// start, every group's source and destination permutation.
template <int g, int MG>
__device__ void run_pair(const PlanArgs& P, const FamCtx& fc, uint8_t* SL, uint8_t* DL, int start,
                         const uint8_t* rperm, int lane, uint64_t top, bool need_x, PairRes* out) {
  constexpr int g2 = g * g, kRow = g2 | 1;   // credit rows padded to an odd word count
  const int G = P.L.G;
  int o[MG][g], nn_[MG][g], ip[MG][g], sig[MG][g], del[MG][g];
  bool own[MG];
#pragma unroll
  for (int r = 0; r < MG; ++r) {
    const int a = lane + 64 * r;
    own[r] = a < G;
#pragma unroll
    for (int m = 0; m < g; ++m) {
      o[r][m] = own[r] ? fc.outT[a * g + m] : 0;
      nn_[r][m] = own[r] ? fc.inT[a * g + m] : 0;
      ip[r][m] = own[r] ? fc.ipos[a * g + m] : -1;
      sig[r][m] = m;
      del[r][m] = m;
    }
  }
  int protect = -1;
  if (start == 0) {
    // canonical binding plus the highest-credit triple, ties to the smallest (t, i, j)
    if (top) {
      const int idx = 0xFFFFFF - (int)(top & 0xFFFFFF);
      const int ts = idx / g2, e = idx - ts * g2;
      const int il = e / g, jl = e - il * g;
      protect = ts;
#pragma unroll
      for (int r = 0; r < MG; ++r) {
        if (!own[r]) continue;
#pragma unroll
        for (int m = 0; m < g; ++m) {
          if (o[r][m] == ts) {
#pragma unroll
            for (int m2 = 0; m2 < g; ++m2)
              if (sig[r][m2] == il) {
                sig[r][m2] = sig[r][m];
                sig[r][m] = il;
              }
          }
          if (nn_[r][m] == ts) {
#pragma unroll
            for (int m2 = 0; m2 < g; ++m2)
              if (del[r][m2] == jl) {
                del[r][m2] = del[r][m];
                del[r][m] = jl;
              }
          }
        }
      }
    }
  } else {
    // independent Fisher-Yates shuffles of every group's sources and
    // destinations, drawn during the credit gather (packed 2 bits per member)
#pragma unroll
    for (int r = 0; r < MG; ++r) {
      if (!own[r]) continue;
      const int a = lane + 64 * r;
      const int ps = rperm[2 * a], pd = rperm[2 * a + 1];
#pragma unroll
      for (int m = 0; m < g; ++m) {
        sig[r][m] = (ps >> (2 * m)) & 3;
        del[r][m] = (pd >> (2 * m)) & 3;
      }
    }
  }
  // Self-binding repair, per group in out-list order: trade destinations with
  // the first other unprotected in-instance, else sources with the first
  // other unprotected out-instance.
#pragma unroll
  for (int r = 0; r < MG; ++r) {
    if (!own[r]) continue;
#pragma unroll
    for (int m = 0; m < g; ++m) {
      const int mi = ip[r][m];
      if (mi < 0 || sig[r][m] != del[r][mi]) continue;
      int partner = -1;
#pragma unroll
      for (int m2 = 0; m2 < g; ++m2)
        if (partner < 0 && nn_[r][m2] != o[r][m] && nn_[r][m2] != protect) partner = m2;
      if (partner >= 0) {
        const int x = del[r][mi];
        del[r][mi] = del[r][partner];
        del[r][partner] = x;
        continue;
      }
#pragma unroll
      for (int m3 = 0; m3 < g; ++m3)
        if (partner < 0 && o[r][m3] != o[r][m] && o[r][m3] != protect) partner = m3;
      if (partner >= 0) {
        const int x = sig[r][m];
        sig[r][m] = sig[r][partner];
        sig[r][partner] = x;
      }
    }
  }
#pragma unroll
  for (int r = 0; r < MG; ++r) {
    if (!own[r]) continue;
#pragma unroll
    for (int m = 0; m < g; ++m) {
      SL[o[r][m]] = (uint8_t)sig[r][m];
      DL[nn_[r][m]] = (uint8_t)del[r][m];
    }
  }
  wave_sync();

  // The credit rows of the owned groups' out- and in-instances do not change
  // during the run: with few enough of them they are read once here and held
  // in registers, and a half-step reads only the other side's assignment.
  constexpr bool kHold = 2 * MG * g * g2 <= 64;
  int32_t hs[kHold ? MG : 1][g][g2], hd[kHold ? MG : 1][g][g2];
  if constexpr (kHold) {
#pragma unroll
    for (int r = 0; r < MG; ++r)
#pragma unroll
      for (int m = 0; m < g; ++m)
#pragma unroll
        for (int e = 0; e < g2; ++e) {
          hs[r][m][e] = fc.H[o[r][m] * kRow + e];
          hd[r][m][e] = fc.H[nn_[r][m] * kRow + e];
        }
  }

  // Alternating Algorithm: source half, then destination half.  A half that
  // changes nothing, other than the very first, leaves a fixed point: the
  // half before it made its own side optimal against this side, which has
  // not moved.  Stopping there gives the same binding as stopping after a
  // whole unchanged sweep, one sweep earlier.
  for (int sweep = 0; sweep < P.i_aa; ++sweep) {
    int changed = 0;
    {
      // every load of the half-step first (destinations and credit rows of all
      // owned groups), then the g! comparisons
      int jl[MG][g];
      int32_t row[MG][g][g2];
#pragma unroll
      for (int r = 0; r < MG; ++r)
#pragma unroll
        for (int m = 0; m < g; ++m) {
          jl[r][m] = DL[o[r][m]];
#pragma unroll
          for (int e = 0; e < g2; ++e) row[r][m][e] = kHold ? hs[r][m][e] : fc.H[o[r][m] * kRow + e];
        }
      // computed for every lane (a lane past the last group reads instance
      // 0's rows and changes nothing): no branch but the guarded writes
#pragma unroll
      for (int r = 0; r < MG; ++r) {
        int32_t h[g][g];
#pragma unroll
        for (int m = 0; m < g; ++m)
#pragma unroll
          for (int il = 0; il < g; ++il) {
            int32_t v = row[r][m][il * g];
#pragma unroll
            for (int jj = 1; jj < g; ++jj) v = jl[r][m] == jj ? row[r][m][il * g + jj] : v;
            h[m][il] = v;
          }
        int32_t cur = 0;
#pragma unroll
        for (int m = 0; m < g; ++m) {
          int32_t v = h[m][0];
#pragma unroll
          for (int i2 = 1; i2 < g; ++i2) v = sig[r][m] == i2 ? h[m][i2] : v;
          cur += v > 0 ? v : 0;   // a self pair counts as zero credit
        }
        int32_t bestv = -1;
        int bp = 0;
#pragma unroll
        for (int p = 0; p < Perms<g>::n; ++p) {
          int32_t v = 0;
#pragma unroll
          for (int m = 0; m < g; ++m) v += h[m][Perms<g>::at(p, m)];
          if (v > bestv) {
            bestv = v;
            bp = p;
          }
        }
        const bool up = own[r] && bestv > cur;
#pragma unroll
        for (int m = 0; m < g; ++m) sig[r][m] = up ? Perms<g>::at(bp, m) : sig[r][m];
        if (up) {
#pragma unroll
          for (int m = 0; m < g; ++m) SL[o[r][m]] = (uint8_t)sig[r][m];
        }
        changed |= up;
      }
    }
    wave_sync();
    if (sweep > 0 && !__any(changed)) break;
    changed = 0;
    {
      int il[MG][g];
      int32_t row[MG][g][g2];
#pragma unroll
      for (int r = 0; r < MG; ++r)
#pragma unroll
        for (int m = 0; m < g; ++m) {
          il[r][m] = SL[nn_[r][m]];
#pragma unroll
          for (int e = 0; e < g2; ++e) row[r][m][e] = kHold ? hd[r][m][e] : fc.H[nn_[r][m] * kRow + e];
        }
#pragma unroll
      for (int r = 0; r < MG; ++r) {
        int32_t h[g][g];
#pragma unroll
        for (int m = 0; m < g; ++m)
#pragma unroll
          for (int jl = 0; jl < g; ++jl) {
            int32_t v = row[r][m][jl];
#pragma unroll
            for (int ii = 1; ii < g; ++ii) v = il[r][m] == ii ? row[r][m][ii * g + jl] : v;
            h[m][jl] = v;
          }
        int32_t cur = 0;
#pragma unroll
        for (int m = 0; m < g; ++m) {
          int32_t v = h[m][0];
#pragma unroll
          for (int j2 = 1; j2 < g; ++j2) v = del[r][m] == j2 ? h[m][j2] : v;
          cur += v > 0 ? v : 0;   // a self pair counts as zero credit
        }
        int32_t bestv = -1;
        int bp = 0;
#pragma unroll
        for (int p = 0; p < Perms<g>::n; ++p) {
          int32_t v = 0;
#pragma unroll
          for (int m = 0; m < g; ++m) v += h[m][Perms<g>::at(p, m)];
          if (v > bestv) {
            bestv = v;
            bp = p;
          }
        }
        const bool up = own[r] && bestv > cur;
#pragma unroll
        for (int m = 0; m < g; ++m) del[r][m] = up ? Perms<g>::at(bp, m) : del[r][m];
        if (up) {
#pragma unroll
          for (int m = 0; m < g; ++m) DL[nn_[r][m]] = (uint8_t)del[r][m];
        }
        changed |= up;
      }
    }
    wave_sync();
    if (!__any(changed)) break;
  }

  // binding score F (Eq. (8)) and the largest lane volume per path class, in units
  int64_t F = 0;
  int32_t xp = 0, xn = 0;
  int jf[MG][g], cf[MG][g];
  int32_t rf[MG][g][g];
#pragma unroll
  for (int r = 0; r < MG; ++r)
#pragma unroll
    for (int m = 0; m < g; ++m) {
      jf[r][m] = DL[o[r][m]];
      cf[r][m] = own[r] ? fc.ocls[(lane + 64 * r) * g + m] : 0;
#pragma unroll
      for (int jl = 0; jl < g; ++jl) {
        if constexpr (kHold) {   // the row is in registers: select the source's part
          int32_t v = hs[r][m][jl];
#pragma unroll
          for (int i2 = 1; i2 < g; ++i2) v = sig[r][m] == i2 ? hs[r][m][i2 * g + jl] : v;
          rf[r][m][jl] = v;
        } else {
          rf[r][m][jl] = fc.H[o[r][m] * kRow + sig[r][m] * g + jl];
        }
      }
    }
#pragma unroll
  for (int r = 0; r < MG; ++r) {
#pragma unroll
    for (int m = 0; m < g; ++m) {
      int32_t x = rf[r][m][0];
#pragma unroll
      for (int jj = 1; jj < g; ++jj) x = jf[r][m] == jj ? rf[r][m][jj] : x;
      x = own[r] && x > 0 ? x : 0;   // a self pair serves nothing
      F += x;
      const bool nic = cf[r][m] == VP_PATH_NIC;
      xn = nic && x > xn ? x : xn;
      xp = !nic && x > xp ? x : xp;
    }
  }
  F = wave_sum(F);
  if (need_x) {   // the lane maxima only serve comparisons between families
    xp = wave_max32(xp);
    xn = wave_max32(xn);
  }
  if (lane == 0) {
    out->F = F;
    out->xmax[0] = xp;
    out->xmax[1] = xn;
  }
}

__device__ inline void set_err(Shared* sh, int code) { atomicCAS(&sh->err, 0, code); }

// Element idx of a global array whose byte offsets stay below 2^32 (checked
// on the host): a 32-bit offset from a wavefront-uniform base, which the
// compiler addresses as scalar base + vector offset.
template <typename T>
__device__ inline T& at32(T* base, uint32_t idx) {
  return *(T*)((char*)base + (uint32_t)(idx * (uint32_t)sizeof(T)));
}

// The first start with the highest binding score F among a family's ns runs
// (F >= 0; enter with F0 = -1).  Four scores are read per round; indices past
// the last read the last again, which never wins a strict comparison.
__device__ inline void best_start(const PairRes* r, int ns, int& s0, int64_t& F0) {
  for (int b = 0; b < ns; b += 4) {
    int64_t f[4];
    int q[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      q[u] = b + u < ns ? b + u : ns - 1;
      f[u] = r[q[u]].F;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (f[u] > F0) {
        F0 = f[u];
        s0 = q[u];
      }
  }
}

// Workgroup barrier that orders LDS only: outstanding global stores of the
// waves are not waited for.
__device__ inline void lds_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0), other counters untouched
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

template <int g, int MG>
__global__ void __launch_bounds__(kPlanThreads) plan_kernel(PlanArgs P) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  // credit rows of the g x g endpoint pairs of an instance, padded to an odd
  // number of words so that the lanes of a wavefront reading consecutive
  // instances' rows fall in different LDS banks
  constexpr int g2 = g * g, kRow = g2 | 1;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const DevCatalogLayout& L = P.L;
  const int N = L.N, Q = L.Q, nn = L.nn, QG = Q * g;
  const int NP = L.J0 + L.J1, NS = P.n_start, FL = L.F0 + L.F1;
  // workgroup b plans matrix b of the batch: every global buffer is offset by b
  const size_t b = blockIdx.x, NN = (size_t)N * N, KN = (size_t)P.k_max * N;
  const int64_t* gD = P.D + b * NN;
  int64_t* gDrem = P.Drem + b * NN;
  int32_t* gfamily = P.family + b * P.k_max;
  int32_t* gdst = P.dst + b * KN;
  int32_t* ginst = P.inst + b * KN;
  int64_t* gbytes = P.bytes + b * KN;
  int64_t* gsend_off = P.send_off ? P.send_off + b * KN : nullptr;
  int64_t* gstream_off = P.stream_off ? P.stream_off + b * KN : nullptr;
  int32_t* grecv_src = P.recv_src ? P.recv_src + b * KN : nullptr;
  constexpr FixedLds FX = fixed_lds((size_t)64 * MG * g);
  Shared* sh = (Shared*)smem;
  int32_t* rinfo = (int32_t*)(smem + FX.rinfo);
  int32_t* agg = (int32_t*)(smem + P.o_agg);         // [q][q2][k] units: k = 0 is A, k > 0 is B_k;
                                                     // then one row of zeros
  // row stride: odd (lanes reading one shift of different rows hit distinct
  // banks) and at least nn + 3 (zero padding for the 4-wide shift unroll)
  const int kS = (nn + 3) | 1;
  uint16_t* terms = (uint16_t*)(smem + P.o_terms);
  int32_t* pfb = (int32_t*)(smem + P.o_pfb);           // [NP][2] local family range
  uint16_t* finfo = (uint16_t*)(smem + P.o_finfo);
  PairRes* pr = (PairRes*)(smem + P.o_pair);
  uint16_t* outT = (uint16_t*)(smem + P.o_outT);
  uint16_t* inT = (uint16_t*)(smem + P.o_inT);
  int8_t* ipos = (int8_t*)(smem + P.o_ipos);
  uint8_t* ocls = smem + P.o_ocls;
  uint8_t* iid = smem + P.o_iid;     // [FC][N] node-local instance id of every instance of the chunk
  int32_t* hp = (int32_t*)(smem + P.o_hp);
  uint32_t* raw = (uint32_t*)(smem + P.o_raw);       // residual of every credit entry (saturating)
  uint8_t* sl = smem + P.o_sl;
  uint8_t* dl = smem + P.o_dl;
  uint8_t* bsl = smem + FX.bsl;
  uint8_t* bdl = smem + FX.bdl;
  uint8_t* bid = smem + FX.bid;
  uint32_t* bx = (uint32_t*)(smem + FX.bx);
  uint32_t* brw = (uint32_t*)(smem + FX.brw);
  uint64_t* topkey = (uint64_t*)(smem + P.o_top);    // [FC] best credit triple of each family in the chunk
  uint16_t* rset = (uint16_t*)(smem + P.o_rset);     // [nS][kMaxRTerms] agg row offsets (zero row past the end)
  uint16_t* psid = (uint16_t*)(smem + P.o_psid);     // [J1] NIC-lane set of each NIC-carrying pattern
  uint64_t* rbest = (uint64_t*)(smem + P.o_rbest);   // [nS] best shift: units << 12 | (4095 - shift)
  int32_t* pbase = (int32_t*)(smem + P.o_pbase);     // [NP] diagonal-block score of each pattern
  // D^rem entry each source rank's lane changed last, and its new value: the
  // next credit gather takes it from here, so no barrier has to wait for the
  // global store (stores of earlier iterations are complete by then).
  uint8_t* rp = smem + P.o_rp;   // [FC][NS][G][2] packed permutations of the shuffled starts
  int32_t* lastj = (int32_t*)(smem + FX.lastj);
  int64_t* sacc = (int64_t*)(smem + FX.sacc);   // [N] bytes each rank has sent so far
  int64_t* lastv = (int64_t*)(smem + FX.lastv);
  const int32_t* cat = P.cat;

  // ---------------------------------------------------------------- prologue
  if (tid == 0) {
    sh->err = 0;
    sh->K = 0;
    sh->total_rem = 0;
    sh->total_units = 0;
    sh->Lmax = 0;
    sh->key = 0;
    sh->huge = 0;
  }
  for (int r = tid; r < N; r += kPlanThreads) {
    const int grp = r / g;
    rinfo[r] = ((grp / Q) << 8) | ((grp % Q) << 4) | (r - grp * g);
  }
  // a diagonal-block term is kept as its count | (q * Q + q2) << 4, the
  // index of its slot pair's A row (the scoring loop reads nothing else); a
  // shift-block term's count is zeroed and each pattern's slots are padded
  // with zeros to a multiple of 8, so no slot needs a bound check
  const int TS8 = (L.TS + 7) & ~7;
  for (int x = tid; x < NP * TS8; x += kPlanThreads) {
    const int p = x / TS8, m = x - p * TS8;
    const int tv = m < L.TS ? cat[L.off_terms + p * L.TS + m] : 0;
    const int cnt = (tv >> 12) == 0 ? (tv & 15) : 0;
    terms[x] = (uint16_t)(cnt | ((((tv >> 8) & 15) * Q + ((tv >> 4) & 15)) << 4));
  }
  for (int p = tid; p < NP; p += kPlanThreads) {
    pfb[2 * p] = cat[L.off_fb + p];
    pfb[2 * p + 1] = cat[L.off_fe + p];
  }
  for (int x = tid; x < FL * QG; x += kPlanThreads) {
    // descriptor word and in-list entry of local family x / QG, index x % QG
    const int lf = x / QG, idx = x - lf * QG;
    const int info = cat[L.off_fam_info + x];
    const int cls = info & 15, ss = (info >> 4) & 15, ds = (info >> 8) & 15;
    int opos = 0;
    for (int m = 0; m < g; ++m)
      if (cat[L.off_fam_out + lf * QG + ss * g + m] == idx) opos = m;
    const bool remote = cls == VP_PATH_NIC && lf >= L.F0;
    int rsame = 0, nother = 0;
    for (int m = 0; m < g; ++m) {
      const int idx2 = cat[L.off_fam_in + lf * QG + ds * g + m];
      const bool r2 = (cat[L.off_fam_info + lf * QG + idx2] & 15) == VP_PATH_NIC && lf >= L.F0;
      if (r2 != remote) ++nother;
      else if (idx2 < idx) ++rsame;
    }
    finfo[x] = (uint16_t)(cls | (ss << 2) | (ds << 5) | (opos << 8) | (rsame << 10) | (nother << 12));
  }
  for (int x = tid; x < kS * (Q * Q + 1); x += kPlanThreads) agg[x] = 0;
  for (int x = tid; x < L.nS * kMaxRTerms; x += kPlanThreads) {
    const int e = cat[L.off_rset + x];
    rset[x] = (uint16_t)((e < 0 ? Q * Q : e) * kS);   // absent terms read the zero row
  }
  for (int x = tid; x < L.J1; x += kPlanThreads) psid[x] = (uint16_t)cat[L.off_psid + x];
  for (int x = tid; x < P.FC; x += kPlanThreads) topkey[x] = 0;
  for (int x = tid; x < N; x += kPlanThreads) {
    lastj[x] = -1;
    sacc[x] = 0;
  }
  int64_t* colsum = (int64_t*)hp;   // the credit area is free during the prologue
  for (int x = tid; x < N; x += kPlanThreads) colsum[x] = 0;
  __syncthreads();

  // one pass over D: validate, copy to D^rem, row / column sums, aggregates.
  // An entry of 2^42 bytes or more is refused before anything is summed: at
  // most 2^20 entries below 2^42 keep every row, column and total sum below
  // 2^62.
  {
    bool bad = false, huge = false;
    int64_t tot = 0, lmax = 0;
    const uint64_t mask = (uint64_t(1) << P.unit_shift) - 1;
    for (int i = wave; i < N; i += kWaves) {
      const int ri = rinfo[i], ni = ri >> 8, qi = (ri >> 4) & 15;
      int64_t rs = 0;
      for (int j = lane; j < N; j += 64) {
        const int64_t v = gD[(size_t)i * N + j];
        const bool divisible = ((uint64_t)v & mask) == 0 &&
                               ((uint64_t)v >> P.unit_shift) * P.odd_inv <= P.odd_lim;
        if (v < 0 || (i == j && v != 0) || !divisible) bad = true;
        if (v >= (int64_t(1) << 42)) huge = true;
        gDrem[(size_t)i * N + j] = v;
        rs += v;
        if (v > 0) {
          const int rj = rinfo[j], nj = rj >> 8, qj = (rj >> 4) & 15;
          int kk = nj - ni;
          if (kk < 0) kk += nn;
          atomicAdd((unsigned long long*)&colsum[j], (unsigned long long)v);
          // exact quotient by the unit: v >> s times the odd part's inverse
          const int32_t vu = (int32_t)(((uint64_t)v >> P.unit_shift) * P.odd_inv);
          atomicAdd(&agg[(qi * Q + qj) * kS + kk], vu);
        }
      }
      rs = wave_sum(rs);
      tot += rs;
      lmax = rs > lmax ? rs : lmax;
    }
    if (bad) set_err(sh, VP_ERR_INVALID_DEMAND);
    if (huge) sh->huge = 1;
    if (lane == 0) {
      atomicAdd((unsigned long long*)&sh->total_rem, (unsigned long long)tot);
      atomicAdd((unsigned long long*)&sh->total_units,
                (unsigned long long)(((uint64_t)tot >> P.unit_shift) * P.odd_inv));
      atomicMax((unsigned long long*)&sh->Lmax, (unsigned long long)lmax);
    }
  }
  __syncthreads();
  {
    int64_t lmax = 0;
    for (int j = tid; j < N; j += kPlanThreads) lmax = colsum[j] > lmax ? colsum[j] : lmax;
    lmax = wave_max(lmax);
    if (lane == 0) atomicMax((unsigned long long*)&sh->Lmax, (unsigned long long)lmax);
  }
  __syncthreads();
  if (tid == 0 && sh->err == 0) {
    const int64_t den = L.bw_max * P.k_target;
    int64_t tau = (sh->Lmax + den - 1) / den;
    if (tau < 1) tau = 1;
    sh->tau = tau;
    for (int c = 0; c < 4; ++c) {
      int64_t cap = tau * L.bw_cls[c] / P.unit * P.unit;
      if (cap < P.unit) cap = P.unit;
      sh->cap[c] = cap;
      sh->capu[c] = (int32_t)(cap / P.unit);
      // credits are int32 bytes below 2^31 and int32 units below 2^27
      if (cap >= (int64_t(1) << 31) || cap / P.unit >= (int64_t(1) << 27)) set_err(sh, VP_ERR_UNSUPPORTED);
    }
    if (sh->huge || sh->total_rem >= (int64_t(1) << 42) || sh->total_units >= (int64_t(1) << 28))
      set_err(sh, VP_ERR_UNSUPPORTED);
  }
  __syncthreads();

  // this thread's first (family, instance) item of a gather and the step
  // between its items, fixed for the plan
  const int g_c0 = tid / N, g_t0 = tid - (tid / N) * N, g_dc = kPlanThreads / N, g_dt = kPlanThreads % N;
  // the per-class caps are plan constants: held in registers
  const int64_t cap_c0 = lane0(sh->cap[0]), cap_c1 = lane0(sh->cap[1]), cap_c2 = lane0(sh->cap[2]),
                cap_c3 = lane0(sh->cap[3]);
  // ---------------------------------------------------------------- loop
  int stamp_it = 0;
  (void)stamp_it;
  while (true) {
    // The loop's exit conditions are read here and tested after the scoring
    // work, which does not depend on them (on the last pass it is wasted),
    // so the read's latency hides behind it.
    const int err_ = sh->err, K_ = sh->K;
    stamp_it = K_;
    VP_STAMP(0);
    const int64_t rem_ = sh->total_rem;

    // Step 1: score every shape; argmax.  A shape (k, p) scores base(p), its
    // diagonal-block terms against A, plus, for k > 0, the sum of B_k over
    // its NIC-lane set.  The shift part depends on p only through that set,
    // so (a) every distinct set finds its best shift (LPS lanes per set,
    // SPT shifts each, ties to the lowest shift) while other threads compute
    // every base(p); (b) one thread per pattern adds its set's best and the
    // block takes the argmax (ties to the lowest canonical shape index).
    {
      const int na = L.nS * P.LPS;
      for (int x = tid; x < na + NP; x += kPlanThreads) {
        if (x < na) {
          const int si = x >> P.LPS_log2, ch = x & (P.LPS - 1);
          const int k0 = 1 + ch * P.SPT, k1 = min(nn, k0 + P.SPT);
          // all loads unconditional and independent: absent terms read the zero row
          int off[kMaxRTerms];
#pragma unroll
          for (int m = 0; m < kMaxRTerms; ++m) off[m] = rset[si * kMaxRTerms + m];
          // sums are never negative: the first shift always takes the lead,
          // and a strict gain keeps the lowest of equal shifts
          int32_t br = -1;
          int bk = 0;
          for (int kb = k0; kb < k1; kb += 4) {
            int32_t r0 = 0, r1 = 0, r2 = 0, r3 = 0;
#pragma unroll
            for (int m0 = 0; m0 < kMaxRTerms; m0 += 4) {
              if (m0 >= P.MRT) break;
#pragma unroll
              for (int m = m0; m < m0 + 4; ++m) {
                const int32_t* row = agg + off[m] + kb;   // rows are zero-padded past nn
                r0 += row[0];
                r1 += row[1];
                r2 += row[2];
                r3 += row[3];
              }
            }
            if (r0 > br) {
              br = r0;
              bk = kb;
            }
            if (kb + 1 < k1 && r1 > br) {
              br = r1;
              bk = kb + 1;
            }
            if (kb + 2 < k1 && r2 > br) {
              br = r2;
              bk = kb + 2;
            }
            if (kb + 3 < k1 && r3 > br) {
              br = r3;
              bk = kb + 3;
            }
          }
          uint64_t bkey = br >= 0 ? ((uint64_t)(uint32_t)br << 12) | (uint64_t)(4095 - bk) : 0;
          // the LPS lanes of a set are adjacent lanes of one wavefront
          for (int o = 1; o < P.LPS; o <<= 1) {
            const uint64_t y = __shfl_xor(bkey, o);
            bkey = y > bkey ? y : bkey;
          }
          if (ch == 0) rbest[si] = bkey;
        } else {
          const int p = x - na;
          const uint16_t* tp = terms + p * TS8;
          // term slots eight at a time up to the longest diagonal part, the
          // slot loads of a group issued together and then their A loads;
          // shift-block and padding slots weigh zero
          int32_t sb = 0;
          for (int m0 = 0; m0 < P.MLT; m0 += 8) {
            int tv[8];
#pragma unroll
            for (int m = 0; m < 8; ++m) tv[m] = tp[m0 + m];
            int32_t av[8];
#pragma unroll
            for (int m = 0; m < 8; ++m) av[m] = agg[__umul24((unsigned)(tv[m] >> 4), (unsigned)kS)];
#pragma unroll
            for (int m = 0; m < 8; ++m) sb += (tv[m] & 15) * av[m];
          }
          pbase[p] = sb;
        }
      }
    }
    VP_STAMP(1);
    if (err_ || rem_ == 0) break;   // the same LDS words for every thread
    if (K_ >= P.k_max) {
      __syncthreads();
      if (tid == 0) set_err(sh, VP_ERR_CAPACITY);
      break;
    }
    // iteration-wide values read from LDS are made wavefront-uniform, so
    // that what is derived from them runs on the scalar unit
    const int K = lane0(K_);
    lds_barrier();
    VP_STAMP(2);
    {
      uint64_t best = 0;
      for (int p = tid; p < NP; p += kPlanThreads) {
        int32_t sc = pbase[p];
        int j = p;
        if (p >= L.J0) {
          const uint64_t rb = rbest[psid[p - L.J0]];
          sc += (int32_t)(rb >> 12);
          j = ((4095 - (int)(rb & 4095)) << 12) | (p - L.J0);   // same order as the canonical shape index
        }
        const uint64_t key = ((uint64_t)(uint32_t)sc << 20) | (uint64_t)(0xFFFFF - j);
        best = key > best ? key : best;
      }
      best = wave_max_u(best);
      if (lane == 0 && best) atomicMax((unsigned long long*)&sh->key, (unsigned long long)best);
    }
    lds_barrier();
    const uint64_t key = (uint64_t)lane0((int64_t)sh->key);
    VP_STAMP(3);
    if ((key >> 20) == 0) {
      __syncthreads();
      if (tid == 0) set_err(sh, VP_ERR_NO_PROGRESS);
      break;
    }
    const int code = 0xFFFFF - (int)(key & 0xFFFFF);
    const int kstar = code >> 12, pstar = kstar ? L.J0 + (code & 4095) : code;
    const int lb = lane0(pfb[2 * pstar]), le = lane0(pfb[2 * pstar + 1]);
    const int fbase = kstar == 0 ? 0 : (kstar - 1) * L.F1;
    const int fb = lb + fbase, fe = le + fbase;
    // best candidate of the iteration so far: each wavefront that writes the
    // winner evaluates the candidates itself (the same reads in the same
    // order), so each holds it in registers and no barrier separates the
    // evaluation from the update
    bool best_valid = false;
    int64_t best_S = 0, best_xm = 0, best_bm = 1;
    int best_f = 0, best_c = 0, best_s = 0, best_chunk = 0;

    // Steps 2-3 over the shape's bucket, FC families at a time.
    int last_cb = fb;
    for (int cb = fb; cb < fe; cb += P.FC) {
      last_cb = cb;
      const int nc = min(P.FC, fe - cb);
      // group lists and credits of every (family, instance)
      {
        const int tot = nc * N;
        int c = g_c0, t = g_t0;
        for (int x = tid; x < tot; x += kPlanThreads) {
          // local family: f - fbase stays inside the pattern's local range
          const int lf = cb - fbase + c;
          const int n = (int)__umulhi((unsigned)t, P.qg_magic), idx = t - n * QG;   // t / QG
          const uint32_t w = finfo[lf * QG + idx];
          const int cl = d_cls(w), a = n * Q + d_ss(w);
          int dn = n;
          if (cl == VP_PATH_NIC && kstar) {
            dn = n + kstar;
            if (dn >= nn) dn -= nn;
          }
          const int d = dn * Q + d_ds(w);
          // rank of t inside the in-list of group d (family order = ascending t)
          const bool remote = cl == VP_PATH_NIC && kstar;
          const bool remote_first = dn >= kstar;   // cross-node sources sit on a lower node
          const int mi = d_rsame(w) + ((remote != remote_first) ? d_nother(w) : 0);
          const int op = d_opos(w);
          // Every global load of the item is issued first, unconditionally:
          // the residuals of its g x g pairs (a self pair's zero entry is
          // read and not used; the value is stale only for the entry the
          // last update changed, which LDS holds) and the instance id, which
          // is only written out with the winner.
          int64_t gv[g][g];
#pragma unroll
          for (int il = 0; il < g; ++il)
#pragma unroll
            for (int jl = 0; jl < g; ++jl) gv[il][jl] = at32(gDrem, (uint32_t)((a * g + il) * N + d * g + jl));
          const int idv = cat[L.off_fam_info + lf * QG + idx];
          int lj[g];
          int64_t lv[g];
#pragma unroll
          for (int il = 0; il < g; ++il) {
            lj[il] = lastj[a * g + il];
            lv[il] = lastv[a * g + il];
          }
          const size_t base = (size_t)c * N;
          outT[base + a * g + op] = (uint16_t)t;
          inT[base + d * g + mi] = (uint16_t)t;
          ocls[base + a * g + op] = (uint8_t)cl;
          ipos[base + a * g + op] = (int8_t)(d == a ? mi : -1);
          const int64_t cap = cl == 0 ? cap_c0 : cl == 1 ? cap_c1 : cl == 2 ? cap_c2 : cap_c3;
          int32_t* h = hp + (base + t) * kRow;
          uint32_t* rw = raw + (base + t) * kRow;
          uint64_t kt = 0;
#pragma unroll
          for (int il = 0; il < g; ++il)
#pragma unroll
            for (int jl = 0; jl < g; ++jl) {
              const int i = a * g + il, j = d * g + jl;
              const int64_t dv = lj[il] == j ? lv[il] : gv[il][jl];
              // min(D^rem, cap) < 2^31 bytes, a multiple of the unit: exact quotient
              const uint32_t vb = (uint32_t)(dv < cap ? dv : cap);
              int32_t v = (int32_t)((vb >> P.unit_shift) * (uint32_t)P.odd_inv);
              uint32_t rv = (uint32_t)(dv < (int64_t)kRawSaturated ? dv : (int64_t)kRawSaturated);
              const uint64_t key = ((uint64_t)(uint32_t)v << 24) | (uint64_t)(0xFFFFFF - (t * g2 + il * g + jl));
              if (i == j) {
                v = kForbiddenU;
                rv = kForbidden;
              } else if (v > 0 && key > kt) {
                kt = key;
              }
              h[il * g + jl] = v;
              rw[il * g + jl] = rv;
            }
          iid[base + t] = (uint8_t)(idv >> 12);
          if (N % 64 == 0) {   // one family per wavefront
            kt = wave_max_u(kt);
            if (lane == 0 && kt) atomicMax((unsigned long long*)&topkey[c], (unsigned long long)kt);
          } else if (kt) {
            atomicMax((unsigned long long*)&topkey[c], (unsigned long long)kt);
          }
          c += g_dc;
          t += g_dt;
          if (t >= N) {
            t -= N;
            ++c;
          }
        }
        VP_STAMP(9);
        // the shuffled starts' permutations (Fisher-Yates on SplitMix64
        // streams keyed by seed, iteration, family, start, group and side):
        // one (family, start) pair and 64 of its groups per wavefront, on the
        // wavefronts the gather leaves idle (on all of them when it leaves
        // none).  The pair's key prefix is uniform over the wavefront and a
        // group's two sides share their key, so a lane draws one group.
        {
          const int pairs = nc * (NS - 1), gb = (L.G + 63) >> 6;
          const int busy = (nc * N + 63) >> 6;
          const int w0 = busy < kWaves ? busy : 0, nw = kWaves - w0;
          for (int blk = lane0(wave) - w0; blk >= 0 && blk < pairs * gb; blk += nw) {
            const int cs = blk / gb, a = (blk - cs * gb) * 64 + lane;
            const int cc = cs / (NS - 1), st = 1 + (cs - cc * (NS - 1));
            uint64_t k3 = P.seed;
            k3 = sm_mix(k3 + kGolden) ^ (uint64_t)K;
            k3 = sm_mix(k3 + kGolden) ^ (uint64_t)(cb + cc);
            k3 = sm_mix(k3 + kGolden) ^ (uint64_t)st;
            if (a < L.G) {
              const uint64_t k5 = sm_mix((sm_mix(k3 + kGolden) ^ (uint64_t)a) + kGolden);
              int packed = 0;
#pragma unroll
              for (int side = 0; side < 2; ++side) {
                uint64_t state = k5 ^ (uint64_t)side;
                int perm[g];
#pragma unroll
                for (int m = 0; m < g; ++m) perm[m] = m;
#pragma unroll
                for (int m = g - 1; m >= 1; --m) {
                  state += kGolden;
                  const int j = (int)(sm_mix(state) % (uint64_t)(m + 1));
                  const int x2 = perm[m];
                  perm[m] = perm[j];
                  perm[j] = x2;
                }
#pragma unroll
                for (int m = 0; m < g; ++m) packed |= perm[m] << (2 * m + 8 * side);
              }
              // byte 2a + side of the pair's entry (little-endian halfword)
              *(uint16_t*)(rp + ((size_t)(cc * NS + st) * L.G + a) * 2) = (uint16_t)packed;
            }
          }
        }
        VP_STAMP(10);
      }
      lds_barrier();
      VP_STAMP(4);
      for (int pi = wave; pi < nc * NS; pi += kWaves) {
        const int c = pi / NS, s = pi - c * NS;
        FamCtx fc{outT + (size_t)c * N, inT + (size_t)c * N, ipos + (size_t)c * N, ocls + (size_t)c * N,
                  hp + (size_t)c * N * kRow, cb + c};
        run_pair<g, MG>(P, fc, sl + (size_t)pi * N, dl + (size_t)pi * N, s, rp + (size_t)pi * L.G * 2, lane,
                        topkey[c], fe - fb > 1, &pr[pi]);
      }
      VP_STAMP(5);
      // full barrier: the previous iteration's D^rem stores are complete
      // before the next gather reads D^rem
      __syncthreads();
      VP_STAMP(6);
      // Evaluate (Eq. (9)-(10)): best start per family, best family overall.
      // Only the wavefronts that write the winner (threads t < N) evaluate.
      if (wave == 1)
        for (int x = lane; x < P.FC; x += 64) topkey[x] = 0;   // for the next gather
      if (wave * 64 < N && fe - fb == 1) {
        // a one-family shape: its best start wins, no utility to compare
        // (every lane reads the same scores)
        int s0 = 0;
        int64_t F0 = -1;
        best_start(pr, NS, s0, F0);
        best_valid = true;
        VP_STAMP(11);
        best_S = F0 * P.unit;
        best_f = cb;
        best_c = 0;
        best_s = s0;
        best_chunk = cb;
      } else if (wave * 64 < N) {
        int64_t S = 0, xm = 0, bm = 1;
        int c = -1, bs = 0;
        for (int cc = lane; cc < nc; cc += 64) {
          int s0 = 0;
          int64_t F0 = -1;
          best_start(pr + cc * NS, NS, s0, F0);
          const PairRes& r = pr[cc * NS + s0];
          int64_t xm2 = 0, bm2 = 1;
          for (int cl = 0; cl < 2; ++cl) {
            const int64_t b = L.bw_cls[cl ? VP_PATH_NIC : VP_PATH_PIX];
            if (r.xmax[cl] * bm2 > xm2 * b) {
              xm2 = r.xmax[cl];
              bm2 = b;
            }
          }
          // Eq. (10) in bytes: served volume and slowest lane
          const int64_t Sb = r.F * P.unit;
          xm2 *= P.unit;
          if (c < 0 || utility_greater(Sb, xm2, bm2, S, xm, bm, P.lambda)) {
            S = Sb;
            xm = xm2;
            bm = bm2;
            c = cc;
            bs = s0;
          }
        }
        // wave argmax under the exact order, ties to the lower family index
        for (int off = nc > 1 ? 32 : 0; off > 0; off >>= 1) {
          const int64_t S2 = __shfl_xor(S, off), xm2 = __shfl_xor(xm, off), bm2 = __shfl_xor(bm, off);
          const int c2 = __shfl_xor(c, off), bs2 = __shfl_xor(bs, off);
          bool take = false;
          if (c2 >= 0) {
            if (c < 0) take = true;
            else if (utility_greater(S2, xm2, bm2, S, xm, bm, P.lambda)) take = true;
            else if (!utility_greater(S, xm, bm, S2, xm2, bm2, P.lambda) && c2 < c) take = true;
          }
          if (take) {
            S = S2;
            xm = xm2;
            bm = bm2;
            c = c2;
            bs = bs2;
          }
        }
        // lane 0 holds the chunk's winner (every lane does after the
        // reduction above): make it uniform
        S = lane0(S);
        xm = lane0(xm);
        bm = lane0(bm);
        c = lane0(c);
        bs = lane0(bs);
        if (!best_valid || utility_greater(S, xm, bm, best_S, best_xm, best_bm, P.lambda)) {
          best_valid = true;
          best_S = S;
          best_xm = xm;
          best_bm = bm;
          best_f = cb + c;
          best_c = c;
          best_s = bs;
          best_chunk = cb;
        }
      }
      if (cb + P.FC < fe) {
        // a later chunk reuses this LDS (and the top keys just cleared): keep
        // the winner's binding and volumes, and wait for every wavefront
        if (best_chunk == cb) {
          const int pi = best_c * NS + best_s;
          const int32_t* H = hp + (size_t)best_c * N * kRow;
          const uint32_t* RW = raw + (size_t)best_c * N * kRow;
          for (int t = tid; t < N; t += kPlanThreads) {
            const uint8_t s_ = sl[(size_t)pi * N + t], d_ = dl[(size_t)pi * N + t];
            bsl[t] = s_;
            bdl[t] = d_;
            bid[t] = iid[(size_t)best_c * N + t];
            const int32_t hx = H[t * kRow + s_ * g + d_];
            bx[t] = (uint32_t)(hx > 0 ? hx : 0);
            brw[t] = RW[t * kRow + s_ * g + d_];
          }
        }
        __syncthreads();
      }
    }

    VP_STAMP(7);
    // Step 4: append E* and subtract X(E*) from D^rem and the aggregates.
    {
      const int f = best_f, k = kstar;
      const int lf = f - fbase;
      const bool live = best_chunk == last_cb;
      const int pi = best_c * NS + best_s;
      const uint8_t* SLp = live ? sl + (size_t)pi * N : bsl;
      const uint8_t* DLp = live ? dl + (size_t)pi * N : bdl;
      const int32_t* H = hp + (size_t)best_c * N * kRow;
      const uint32_t* RW = raw + (size_t)best_c * N * kRow;
      for (int t = tid; t < N; t += kPlanThreads) {
        const int n = (int)__umulhi((unsigned)t, P.qg_magic), idx = t - n * QG;   // t / QG
        const uint32_t w = finfo[lf * QG + idx];
        const int cl = d_cls(w), ss = d_ss(w), ds = d_ds(w);
        int dn = n;
        if (cl == VP_PATH_NIC && k) {
          dn = n + k;
          if (dn >= nn) dn -= nn;
        }
        const int s_ = SLp[t], d_ = DLp[t];
        const int i = (n * Q + ss) * g + s_, j = (dn * Q + ds) * g + d_;
        int32_t xu = live ? H[t * kRow + s_ * g + d_] : (int32_t)bx[t];   // units
        xu = xu > 0 ? xu : 0;   // a self pair serves nothing
        // the unit is below 2^31 (a cap of at least one unit fits 31 bits)
        const int64_t x = (int64_t)((uint64_t)(uint32_t)xu * (uint32_t)P.unit);
        const uint32_t rv = live ? RW[t * kRow + s_ * g + d_] : brw[t];
        VP_STAMP(12);
        const uint32_t o = (uint32_t)(K * N + i);
        at32(gdst, o) = j;
        at32(ginst, o) = live ? iid[(size_t)best_c * N + t] : bid[t];
        at32(gbytes, o) = x;
        if (grecv_src) at32(grecv_src, (uint32_t)(K * N + j)) = i;   // pi_k is a permutation
        // A residual that did not fit its 32-bit copy is reloaded from
        // D^rem.  Every use of such a reload stays inside its own branch,
        // whose stores are relaxed atomic ones so that they are not merged
        // with the common path's: a use after the branches would make the
        // common path wait for every store issued so far (the wait counter
        // covers stores as well).
        const bool sat = rv >= kRawSaturated;
        if (gsend_off) {
          // Sec. 5 buffer layout: where this lane's slice sits in rank i's
          // send buffer and in its stream to j (bytes sent there before:
          // D[i][j] minus the residual before this step; D[i][j] is added by
          // stream_off_kernel after the plan, which keeps its load off this
          // loop's critical path)
          at32(gsend_off, o) = sacc[i];
          if (__builtin_expect(!sat, 1))
            at32(gstream_off, o) = -(int64_t)rv;
          else
            __hip_atomic_store(&at32(gstream_off, o), -at32(gDrem, (uint32_t)(i * N + j)), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
          sacc[i] += x;
        }
        VP_STAMP(13);
        if (xu > 0) {
          int64_t* dp = &at32(gDrem, (uint32_t)(i * N + j));
          if (__builtin_expect(!sat, 1)) {
            const int64_t nv = (int64_t)rv - x;
            *dp = nv;
            lastv[i] = nv;
          } else {
            const int64_t nv = *dp - x;
            __hip_atomic_store(dp, nv, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(&lastv[i], nv, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
          }
          lastj[i] = j;
          int kk = dn - n;
          if (kk < 0) kk += nn;
          atomicAdd(&agg[(ss * Q + ds) * kS + kk], -xu);
        }
      }
      if (tid == 0) {
        gfamily[K] = f;
        if (best_S == 0) {
          set_err(sh, VP_ERR_NO_PROGRESS);
        } else {
          sh->total_rem -= best_S;
          sh->K = K + 1;
        }
        sh->key = 0;
      }
      VP_STAMP(14);
      // LDS-only barrier: the global stores above need not land before the
      // next scoring pass (which reads LDS only); the full barrier after it
      // orders them before the next gather reads D^rem.
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0), other counters untouched
      __builtin_amdgcn_s_barrier();
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      VP_STAMP(8);
    }
  }

  if (tid == 0) {
    P.K[b] = sh->K;
    if (P.tau) P.tau[b] = sh->err == VP_ERR_INVALID_DEMAND ? 0 : sh->tau;
    if (sh->err) atomicCAS(P.status + b, 0, sh->err);
  }
}

// Stream offsets, completed after the plan: the planner stored minus the
// pair's residual before each step, and the bytes of the pair sent before it
// are D[i][j] plus that (Sec. 5 buffer layout).  Block row b of the grid
// handles matrix b of the batch; its steps k < K[b] only.
__global__ void __launch_bounds__(256) stream_off_kernel(const int64_t* __restrict__ D, const int32_t* __restrict__ K,
                                                         const int32_t* __restrict__ dst, int64_t* stream_off, int N,
                                                         int k_max) {
  const size_t b = blockIdx.y, NN = (size_t)N * N, KN = (size_t)k_max * N;
  const int64_t* Db = D + b * NN;
  const int32_t* db = dst + b * KN;
  int64_t* sb = stream_off + b * KN;
  const size_t n = (size_t)K[b] * N;
  for (size_t x = (size_t)blockIdx.x * 256 + threadIdx.x; x < n; x += (size_t)gridDim.x * 256) {
    const size_t i = x % (size_t)N;
    const int j = db[x];   // every lane of a step is written; checked all the same
    if ((unsigned)j < (unsigned)N) sb[x] += Db[i * N + j];
  }
}

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

template <int g, int MG>
vp_status launch_t(const PlanArgs& P, size_t lds, hipStream_t st) {
  auto kern = plan_kernel<g, MG>;
  if (hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) !=
      hipSuccess)
    return set_error(VP_ERR_HIP, "cannot raise the planner's LDS limit");
  hipLaunchKernelGGL(kern, dim3((unsigned)P.batch), dim3(kPlanThreads), lds, st, P);
  if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "planner launch failed");
  if (P.stream_off) {
    const size_t KN = (size_t)P.k_max * P.L.N;
    const unsigned bx = (unsigned)std::max<size_t>(1, std::min<size_t>((KN + 255) / 256, 2048 / (size_t)P.batch));
    hipLaunchKernelGGL(stream_off_kernel, dim3(bx, (unsigned)P.batch), dim3(256), 0, st, P.D, P.K, P.dst,
                       P.stream_off, P.L.N, P.k_max);
    if (hipGetLastError() != hipSuccess) return set_error(VP_ERR_HIP, "stream offset launch failed");
  }
  return VP_OK;
}

template <int g>
vp_status launch_g(const PlanArgs& P, size_t lds, hipStream_t st, int gpl) {
  if (gpl <= 1) return launch_t<g, 1>(P, lds, st);
  if (gpl <= 2) return launch_t<g, 2>(P, lds, st);
  if (gpl <= 4) return launch_t<g, 4>(P, lds, st);
  return launch_t<g, 8>(P, lds, st);
}

}  // namespace

// ------------------------------------------------- library-owned residual

// vp_plan_noalloc keeps the residual D^rem in this array instead of a
// caller's workspace: one copy per device, held until the process ends,
// room for kStaticRanks ranks.  Host code never passes the array's name to
// a kernel: it passes the device address looked up below.
static __device__ __align__(256) int64_t scratch[(size_t)kStaticRanks * kStaticRanks];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};
}  // namespace

vp_status static_residual(int32_t n_ranks, void** out) {
  if (n_ranks < 1 || n_ranks > kStaticRanks)
    return set_error(VP_ERR_UNSUPPORTED, "vp_plan_noalloc plans at most " + std::to_string(kStaticRanks) +
                                             " ranks (its residual is a fixed device array)");
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return set_error(VP_ERR_HIP, "hipGetDevice failed");
  if (dev < 0 || dev >= kMaxDevices) return set_error(VP_ERR_UNSUPPORTED, "device index too large");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_addr[dev]) {
    // once per device, with that device current: its copy's address
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return set_error(VP_ERR_HIP, std::string("hipGetSymbolAddress of the static residual failed: ") +
                                       hipGetErrorString(e));
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return VP_OK;
}

vp_status launch_plan(const PlanLaunch& a, void* stream) {
  const vp_catalog& c = *a.cat;
  const DevCatalogLayout& L = c.lay;
  const int N = L.N, g = L.g, g2 = g * g, NS = a.p.n_start, NP = L.J0 + L.J1, FL = L.F0 + L.F1;
  const int QG = L.Q * g;
  if (L.J0 > 4095 || L.J1 > 4095 || L.nn > 255) return set_error(VP_ERR_UNSUPPORTED, "catalog too large");
  if (QG > kMaxQG || L.Q > 8 || g > 4) return set_error(VP_ERR_UNSUPPORTED, "too many lanes per node");
  if (N > 65535 || L.G > 64 * 8) return set_error(VP_ERR_UNSUPPORTED, "too many ranks for the planner");
  if (L.n_inst > 256) return set_error(VP_ERR_UNSUPPORTED, "too many node-local instances");
  // the kernel addresses one matrix's schedule and residual with 32-bit byte offsets
  if ((uint64_t)a.p.k_max * (uint64_t)N * 8 >= (uint64_t(1) << 32))
    return set_error(VP_ERR_UNSUPPORTED, "k_max * N too large for the planner");
  int hmax = 1, mlt = 0, mrt = 0;
  for (int p = 0; p < NP; ++p) {
    hmax = std::max(hmax, c.pat_fe[p] - c.pat_fb[p]);
    int nl = 0;
    for (int v : c.patL[p]) nl += v != 0;
    if (nl > kMaxLTerms) return set_error(VP_ERR_UNSUPPORTED, "too many intra-node lane classes");
    mlt = std::max(mlt, nl);
    int nr = 0;   // cross-node lanes (a slot pair counts once per lane: several NICs per switch)
    for (int v : c.patR[p]) nr += v;
    if (nr > kMaxRTerms) return set_error(VP_ERR_UNSUPPORTED, "too many NIC lanes in one pattern");
    mrt = std::max(mrt, nr);
  }

  PlanArgs P{};
  P.cat = (const int32_t*)c.dev;
  P.L = L;
  P.D = a.demand;
  P.Drem = a.drem;
  P.k_target = a.p.k_target;
  P.lambda = a.p.lambda_ns;
  P.unit = a.p.unit_bytes;
  P.seed = a.p.seed;
  // divisibility by unit = 2^s * odd: low s bits clear and (v >> s) * odd^-1 <= (2^64-1)/odd
  uint64_t u = (uint64_t)a.p.unit_bytes;
  int s = 0;
  while (!(u & 1)) {
    u >>= 1;
    ++s;
  }
  uint64_t inv = u;
  for (int it = 0; it < 6; ++it) inv *= 2 - u * inv;
  P.unit_shift = s;
  P.odd_inv = inv;
  P.odd_lim = ~uint64_t(0) / u;
  P.n_start = NS;
  P.MLT = mlt;
  P.MRT = mrt;
  P.i_aa = a.p.i_aa;
  P.k_max = a.p.k_max;
  // shift chunks per NIC-carrying pattern: enough items to occupy every thread
  // shift scoring: about 8 shifts per lane, lanes per set a power of two
  {
    const int shifts = std::max(1, L.nn - 1);
    int lps = 1;
    while (lps < 64 && lps * 8 < shifts) lps <<= 1;
    P.LPS = lps;
    P.SPT = (shifts + lps - 1) / lps;
    P.qg_magic = (uint32_t)(((uint64_t(1) << 32) + (uint64_t)QG - 1) / (uint64_t)QG);
    P.LPS_log2 = 0;
    while ((1 << P.LPS_log2) < lps) ++P.LPS_log2;
  }
  P.K = a.K;
  P.family = a.family;
  P.dst = a.dst;
  P.inst = a.inst;
  P.bytes = a.bytes;
  P.tau = a.tau;
  P.send_off = a.send_off;
  P.stream_off = a.stream_off;
  P.recv_src = a.recv_src;
  P.status = a.status;
  P.batch = a.batch;

  // the per-rank arrays at the instantiation's fixed offsets first
  const int gpl = (L.G + 63) / 64;
  const int MG = gpl <= 1 ? 1 : gpl <= 2 ? 2 : gpl <= 4 ? 4 : 8;
  size_t o = fixed_lds((size_t)64 * MG * g).end;
  auto take = [&](int32_t* field, size_t bytes) {
    *field = (int32_t)o;
    o = align_up(o + bytes, 16);
  };
  take(&P.o_agg, (size_t)((L.nn + 3) | 1) * (L.Q * L.Q + 1) * 4);
  take(&P.o_terms, (size_t)NP * ((L.TS + 7) & ~7) * 2);
  take(&P.o_pfb, (size_t)NP * 8);
  take(&P.o_finfo, (size_t)FL * QG * 2);
  take(&P.o_rset, (size_t)L.nS * kMaxRTerms * 2);
  take(&P.o_psid, (size_t)L.J1 * 2);
  take(&P.o_rbest, (size_t)L.nS * 8);
  take(&P.o_pbase, (size_t)NP * 4);
  const size_t fixed = o;
  const size_t per_fam = align_up((size_t)NS * sizeof(PairRes), 16) + 2 * align_up((size_t)N * 2, 16) +
                         3 * align_up((size_t)N, 16) + 2 * (size_t)N * (g2 | 1) * 4 + 2 * align_up((size_t)NS * N, 16) + 16 +
                         align_up((size_t)NS * L.G * 2, 16);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return set_error(VP_ERR_HIP, "hipGetDevice failed");
  int lds_max = 0;
  if (hipDeviceGetAttribute(&lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess)
    return set_error(VP_ERR_HIP, "hipDeviceGetAttribute failed");
  const size_t budget = (size_t)lds_max;
  if (fixed + per_fam > budget) return set_error(VP_ERR_UNSUPPORTED, "plan state does not fit in LDS");
  int FC = (int)std::min<size_t>((size_t)std::min(hmax, 64), (budget - fixed) / per_fam);
  FC = std::max(FC, 1);
  P.FC = FC;
  take(&P.o_pair, (size_t)FC * NS * sizeof(PairRes));
  take(&P.o_outT, (size_t)FC * N * 2);
  take(&P.o_inT, (size_t)FC * N * 2);
  take(&P.o_ipos, (size_t)FC * N);
  take(&P.o_ocls, (size_t)FC * N);
  take(&P.o_iid, (size_t)FC * N);
  take(&P.o_hp, std::max((size_t)FC * N * (g2 | 1) * 4, (size_t)N * 8));   // also the prologue's column sums
  take(&P.o_raw, (size_t)FC * N * (g2 | 1) * 4);
  take(&P.o_sl, (size_t)FC * NS * N);
  take(&P.o_dl, (size_t)FC * NS * N);
  take(&P.o_top, (size_t)FC * 8);
  take(&P.o_rp, (size_t)FC * NS * L.G * 2);
  if (o > budget) return set_error(VP_ERR_UNSUPPORTED, "plan state does not fit in LDS");

  hipStream_t st = (hipStream_t)stream;
  switch (g) {
    case 2: return launch_g<2>(P, o, st, gpl);
    case 3: return launch_g<3>(P, o, st, gpl);
    case 4: return launch_g<4>(P, o, st, gpl);
  }
  return set_error(VP_ERR_UNSUPPORTED, "gpus_per_switch must be 2, 3 or 4");
}

}  // namespace vp

#ifdef VP_PHASE_STAMPS
// Reader of the phase stamps of the last plan (stamped builds only).
extern "C" int vp_phase_stamps_read(unsigned long long* out) {
  return (int)hipMemcpyFromSymbol(out, HIP_SYMBOL(vp::g_phase_stamps), sizeof(unsigned long long) * 4096 * 16);
}
#endif
