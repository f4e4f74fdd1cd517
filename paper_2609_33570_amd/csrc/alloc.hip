// Joint H/L/R recovery allocation on gfx950 (Sec. 3.4 Eq. joint-allocation,
// solved as in App. B.2 Eqs. allocation-grid, allocation-integer-costs and
// allocation-dp, with the available actions of App. B.3 Eq.
// available-recovery-actions).
//
// Each unit u takes one action in {R, H, L}: R (recompute) is the baseline
// with zero utility, memory and risk; H keeps the activation (utility tau_h,
// memory dm_h, risk 0); L keeps its low-precision codes (tau_l, dm_l, risk
// psi_u).  Memory and risk costs are rounded up to integer steps of the
// budgets (N_B and N_delta intervals), and the dynamic programme
//   F_i(j, k) = max over available a of F_{i-1}(j - b_i(a), k - r_i(a)) + tau_i(a)
// runs over the (N_B + 1) x (N_delta + 1) grid of exact integer costs.
//
// Mapping.  One launch per pair of units updates the whole grid, one thread
// per cell (rows k of risk cost, columns j of memory cost, a row padded to a
// multiple of 64 cells so that a wave covers 64 consecutive cells of one row;
// each XCD takes one contiguous band of cells).  Each cell forms the first
// unit's value at itself and at the two cells the second unit's actions
// shift it to, from up to nine cells of the table before the pair (fp64, all
// in the 256 MB infinity cache for grids up to a few thousand squared), and
// writes the value after the pair; the chosen action (2 bits) of each unit is
// gathered across the wave with two ballots and stored as two 64-bit masks
// per 64 cells, so the backtracking record of a 1025 x 1025 grid is 279 KB
// per unit.  A reduction kernel then finds the best terminal cell, one wave
// backtracks through the records (four units per round trip), and one wave
// sums the chosen costs in unit order.
//
// Every value is produced by the same fp64 operations in the same order as
// a plain sequential implementation (one addition per unit along a path,
// comparisons with the fixed tie rules), so actions and totals are exact.
#include <math.h>

#include "device_common.hpp"
#include "hilore_internal.hpp"

#pragma clang fp contract(off)

namespace hilore {
namespace {

constexpr int kActR = 0, kActH = 1, kActL = 2;
constexpr int kDpThreads = 256;
constexpr int kPartials = 1024;  // workgroups of the terminal reduction
constexpr int kFinalThreads = 1024;
#ifndef HILORE_DP_GROUP
#define HILORE_DP_GROUP 2
#endif
constexpr int kDpGroup = HILORE_DP_GROUP;  // units per DP launch (1 .. 4)

// Availability of a non-R action (App. B.3 Eq. available-recovery-actions;
// non-R actions with non-positive utility are excluded, App. B.2): verified,
// allowed by the retained representation q (H keeps everything, L excludes
// H, R allows only R), and finite non-negative costs.
__device__ bool action_ok(int act, uint8_t q, uint8_t verified, double tau, double dm,
                          double risk) {
  if (((verified >> act) & 1u) == 0) return false;
  if (q == kActL && act == kActH) return false;
  if (q != kActH && q != kActL) return false;
  if (!(tau > 0.0) || !isfinite(tau)) return false;
  if (!(dm >= 0.0) || !isfinite(dm)) return false;
  if (!(risk >= 0.0) || !isfinite(risk)) return false;
  return true;
}

// Integer cost on a grid of n intervals over `budget` (Eq.
// allocation-integer-costs): ceil(cost / h) with h = budget / n, or n + 1
// (does not fit) beyond n; with a zero budget only a zero cost fits.
__device__ int64_t grid_cost(double cost, double budget, int n) {
  if (!(budget > 0.0)) return cost == 0.0 ? 0 : (int64_t)n + 1;
  const double h = budget / (double)n;
  const double c = ceil(cost / h);
  return c > (double)n ? (int64_t)n + 1 : (int64_t)c;
}

__global__ void costs_kernel(const AllocArgs a, AllocUnitCost *uc) {
  const int u = blockIdx.x * blockDim.x + threadIdx.x;
  if (u >= a.U) return;
  const uint8_t q = a.q[u], v = a.verified[u];
  int ok_h = action_ok(kActH, q, v, a.tau_h[u], a.dm_h[u], 0.0);
  int ok_l = action_ok(kActL, q, v, a.tau_l[u], a.dm_l[u], a.psi[u]) && a.delta_b > 0.0;
  const int64_t b_h = ok_h ? grid_cost(a.dm_h[u], a.m_res, a.n_b) : 0;
  const int64_t b_l = ok_l ? grid_cost(a.dm_l[u], a.m_res, a.n_b) : 0;
  const int64_t r_l = ok_l ? grid_cost(a.psi[u], a.delta_b, a.n_d) : 0;
  if (b_h > a.n_b) ok_h = 0;
  if (b_l > a.n_b || r_l > a.n_d) ok_l = 0;
  AllocUnitCost c;
  c.ok_h = ok_h;
  c.ok_l = ok_l;
  c.b_h = (int32_t)b_h;
  c.b_l = (int32_t)b_l;
  c.r_l = (int32_t)r_l;
  c.reach = 0;  // set by reach_kernel
  c.tau_h = a.tau_h[u];
  c.tau_l = a.tau_l[u];
  uc[u] = c;
}

// Memory cost reach after each unit: the running sum, in unit order, of the
// largest memory cost of each unit's available actions, capped at KB - 1
// (integers, one workgroup: a scan per chunk of 1024 units plus a carry).
// No state after unit i has a memory cost above uc[i].reach.
constexpr int kReachThreads = 1024;
__global__ __launch_bounds__(kReachThreads) void reach_kernel(AllocUnitCost *uc, int U, int KB) {
  __shared__ int part[kReachThreads];
  const int tid = (int)threadIdx.x;
  int carry = 0;
  for (int base = 0; base < U; base += kReachThreads) {
    const int i = base + tid;
    int v = 0;
    if (i < U) {
      const AllocUnitCost c = uc[i];
      v = max(c.ok_h ? c.b_h : 0, c.ok_l ? c.b_l : 0);  // each at most KB
    }
    part[tid] = v;
    __syncthreads();
    for (int off = 1; off < kReachThreads; off <<= 1) {
      const int t = tid >= off ? part[tid - off] : 0;
      __syncthreads();
      part[tid] += t;  // at most 1024 * KB: no overflow for KB <= 4097
      __syncthreads();
    }
    if (i < U) uc[i].reach = min(KB - 1, carry + part[tid]);
    carry = min(KB, carry + part[kReachThreads - 1]);
    __syncthreads();
  }
}

// F_0: 0 at (0, 0), -inf elsewhere (padding cells included), and the second
// table all -inf: a DP launch skips the waves whose cells lie beyond the
// memory cost reach, which must then read as unreachable in either table.
__global__ void init_kernel(double *f0, double *f1, int64_t cells) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < cells) {
    f0[i] = i == 0 ? 0.0 : -INFINITY;
    f1[i] = -INFINITY;
  }
}

// F_i(j, k) of one unit of Eq. allocation-dp from the previous table: the
// actions R, H, L in this order, each replacing the incumbent only when
// strictly larger (the within-state tie rule); `act` receives the chosen
// action.  The caller guarantees 0 <= j < KB and 0 <= k; padding cells
// (j >= KB) stay -inf.
__device__ __forceinline__ double unit_value(const double *__restrict__ prev,
                                             const AllocUnitCost &c, int64_t cell, int j, int k,
                                             int S, int &act) {
  double best = prev[cell];
  act = kActR;
  if (c.ok_h && c.b_h <= j) {
    const double v = prev[cell - c.b_h] + c.tau_h;
    if (v > best) {
      best = v;
      act = kActH;
    }
  }
  if (c.ok_l && c.b_l <= j && c.r_l <= k) {
    const double v = prev[cell - (int64_t)c.r_l * S - c.b_l] + c.tau_l;
    if (v > best) {
      best = v;
      act = kActL;
    }
  }
  return best;
}

// F after the units c[0 .. N-1] (applied in order to the table `prev`) at
// cell (j, k), by the rule of Eq. allocation-dp for the last unit applied to
// the values after the first N - 1 at the cells its actions shift (j, k) to,
// down to unit_value on `prev`.  Every value is formed by the same fp64
// additions and comparisons, in the same order, as N single-unit launches
// would form it.  With `acts`, acts[m] receives unit m's action at (j, k)
// itself (the chain through the unshifted cell), i.e. its record there.
template <int N>
__device__ __forceinline__ double chain_value(const double *__restrict__ prev,
                                              const AllocUnitCost *c, int64_t cell, int j, int k,
                                              int S, int *acts) {
  if constexpr (N == 1) {
    int a;
    const double v = unit_value(prev, c[0], cell, j, k, S, a);
    if (acts) acts[0] = a;
    return v;
  } else {
    double best = chain_value<N - 1>(prev, c, cell, j, k, S, acts);
    int act = kActR;
    const AllocUnitCost &u = c[N - 1];
    if (u.ok_h && u.b_h <= j) {
      const double v =
          chain_value<N - 1>(prev, c, cell - u.b_h, j - u.b_h, k, S, nullptr) + u.tau_h;
      if (v > best) {
        best = v;
        act = kActH;
      }
    }
    if (u.ok_l && u.b_l <= j && u.r_l <= k) {
      const double v = chain_value<N - 1>(prev, c, cell - (int64_t)u.r_l * S - u.b_l,
                                          j - u.b_l, k - u.r_l, S, nullptr) +
                       u.tau_l;
      if (v > best) {
        best = v;
        act = kActL;
      }
    }
    if (acts) acts[N - 1] = act;
    return best;
  }
}

// N consecutive units of Eq. allocation-dp in one launch: each cell reads up
// to 3^N cells of the table before the group (the shifted ones mostly from
// the cache) and writes the table after it and the records of all N units,
// bit for bit what N launches of one unit each would write; the tables in
// between are never stored.
template <int N>
__global__ __launch_bounds__(kDpThreads) void dpn_kernel(const double *__restrict__ prev,
                                                          double *__restrict__ cur,
                                                          uint64_t *__restrict__ pred,
                                                          size_t pred_words_per_unit,
                                                          const AllocUnitCost *__restrict__ uc,
                                                          int KB, int KD, int S) {
  const int n = (int)gridDim.x, x = (int)blockIdx.x & 7, q = n >> 3, rem = n & 7;
  const int bid = x * q + (x < rem ? x : rem) + ((int)blockIdx.x >> 3);
  const int64_t cell = (int64_t)bid * kDpThreads + threadIdx.x;
  const int k = (int)(cell / S), j = (int)(cell % S);
  if (k >= KD) return;  // whole waves: S and the grid are multiples of 64
  AllocUnitCost c[N];
#pragma unroll
  for (int m = 0; m < N; ++m) c[m] = uc[m];
  // A wave (64 consecutive cells of one row) wholly beyond the memory cost
  // reach after the group holds only unreachable states: they stay -inf in
  // both tables, and no path the backtrack follows passes through them, so
  // neither their values nor their records are written.
  if (__builtin_amdgcn_readfirstlane(j) > c[N - 1].reach) return;
  int acts[N];
#pragma unroll
  for (int m = 0; m < N; ++m) acts[m] = kActR;
  double best = -INFINITY;
  if (j < KB) best = chain_value<N>(prev, c, cell, j, k, S, acts);
  cur[cell] = best;
  const int64_t w = cell / kWave;  // 64-cell chunk of this wave
#pragma unroll
  for (int m = 0; m < N; ++m) {
    const uint64_t lo = __ballot(acts[m] & 1), hi = __ballot(acts[m] >> 1);
    if ((threadIdx.x & (kWave - 1)) == 0) {
      pred[m * pred_words_per_unit + 2 * w] = lo;
      pred[m * pred_words_per_unit + 2 * w + 1] = hi;
    }
  }
}

// The better of two terminal candidates: larger value, then the earlier cell
// in (risk cost, memory cost) order, which is lower risk, then lower memory.
__device__ __forceinline__ bool better(double v, int64_t i, double bv, int64_t bi) {
  return v > bv || (v == bv && i < bi);
}

struct Best {
  double v;
  int64_t i;
};

template <int THREADS>
__device__ Best block_best(Best b) {
  __shared__ double sv[THREADS];
  __shared__ int64_t si[THREADS];
  sv[threadIdx.x] = b.v;
  si[threadIdx.x] = b.i;
  __syncthreads();
  for (int off = THREADS / 2; off > 0; off >>= 1) {
    if ((int)threadIdx.x < off && better(sv[threadIdx.x + off], si[threadIdx.x + off],
                                         sv[threadIdx.x], si[threadIdx.x])) {
      sv[threadIdx.x] = sv[threadIdx.x + off];
      si[threadIdx.x] = si[threadIdx.x + off];
    }
    __syncthreads();
  }
  return Best{sv[0], si[0]};
}

__global__ __launch_bounds__(kDpThreads) void terminal_partial_kernel(const double *f,
                                                                       int64_t cells,
                                                                       Best *partial) {
  Best b{-INFINITY, INT64_MAX};
  for (int64_t i = (int64_t)blockIdx.x * kDpThreads + threadIdx.x; i < cells;
       i += (int64_t)gridDim.x * kDpThreads) {
    const double v = f[i];
    if (better(v, i, b.v, b.i)) b = Best{v, i};
  }
  b = block_best<kDpThreads>(b);
  if (threadIdx.x == 0) partial[blockIdx.x] = b;
}

// Action of unit `unit` recorded at cell (j, k).
__device__ __forceinline__ int record(const uint64_t *pred, int64_t unit, int64_t k, int64_t j,
                                      int KD, int64_t chunks) {
  const int64_t w = (unit * KD + k) * chunks + j / kWave;
  const int bit = (int)(j % kWave);
  return (int)((pred[2 * w] >> bit) & 1u) | ((int)((pred[2 * w + 1] >> bit) & 1u) << 1);
}

__device__ __forceinline__ int lane_int(int v, int lane) {
  return __builtin_amdgcn_readlane(v, lane);
}

// Backtracking, one wave.  The record of unit i at the current cell decides
// where the record of unit i - 1 is read, so a walk of one unit per step is
// a chain of dependent loads.  Each round trip instead loads the records of
// units i .. i - 3 at every cell the path can reach from the current one
// (1 + 3 + 9 + 27 = 40 cells, one lane each; lane 1 + 3 + ... + 3^(d-1) + p
// holds the record of unit i - d after the actions whose base-3 digits,
// unit i first, spell p; actions R, H, L are 0, 1, 2) and resolves the four
// actions from registers.  Lanes 0..3 carry the costs of units i .. i - 3
// and fetch those of the next four units during the same round trip.
constexpr int kLookUnits = 4;
constexpr int kLookLanes = 40;

__global__ __launch_bounds__(kFinalThreads) void terminal_backtrack_kernel(
    const AllocArgs a, const Best *partial, int n_partial, const uint64_t *pred,
    const AllocUnitCost *uc, int S, int KD) {
  Best b{-INFINITY, INT64_MAX};
  for (int p = threadIdx.x; p < n_partial; p += kFinalThreads)
    if (better(partial[p].v, partial[p].i, b.v, b.i)) b = partial[p];
  b = block_best<kFinalThreads>(b);
  if (threadIdx.x >= kWave) return;
  const int lane = (int)threadIdx.x;
  int64_t k = b.i / S, j = b.i % S;
  if (lane == 0) {
    a.jk[0] = j;
    a.jk[1] = k;
    a.totals[0] = b.v;
  }
  const int64_t chunks = S / kWave;
  // this lane's depth d and path p, and the base-3 digits of p (unit i's
  // action first)
  const int d = lane == 0 ? 0 : lane < 4 ? 1 : lane < 13 ? 2 : 3;
  const int p = lane - (d == 0 ? 0 : d == 1 ? 1 : d == 2 ? 4 : 13);
  int digit[3];
  {
    int rest = p, pw = d == 3 ? 9 : d == 2 ? 3 : 1;
#pragma unroll
    for (int m = 0; m < 3; ++m) {
      digit[m] = m < d ? rest / pw : kActR;
      if (m < d) {
        rest -= digit[m] * pw;
        pw /= 3;
      }
    }
  }
  // Every load below is issued unconditionally (a lane with nothing to load
  // reads a valid dummy address and discards the value), so that no branch
  // forces a wait: the costs of the next four units are waited for only in
  // the next round trip, and the record load is the one latency per trip.
  const bool cost_lane = lane < kLookUnits;
  auto load_costs = [&](int unit, int &bh, int &bl, int &rl) {
    const bool ok = cost_lane && unit - lane >= 0;
    const AllocUnitCost &c = uc[ok ? unit - lane : 0];
    const int h = c.b_h, l = c.b_l, r = c.r_l;
    bh = ok ? h : 0;
    bl = ok ? l : 0;
    rl = ok ? r : 0;
  };
  int bh, bl, rl;
  load_costs(a.U - 1, bh, bl, rl);
  for (int i = a.U - 1; i >= 0; i -= kLookUnits) {
    int nbh, nbl, nrl;
    load_costs(i - kLookUnits, nbh, nbl, nrl);
    // the cell of this lane's record: the current cell minus the costs of
    // the actions its path takes at units i .. i - d + 1
    int64_t jj = j, kk = k;
#pragma unroll
    for (int m = 0; m < 3; ++m) {
      const int ubh = lane_int(bh, m), ubl = lane_int(bl, m), url = lane_int(rl, m);
      if (digit[m] == kActH) jj -= ubh;
      if (digit[m] == kActL) {
        jj -= ubl;
        kk -= url;
      }
    }
    const bool rec = lane < kLookLanes && i - d >= 0 && jj >= 0 && kk >= 0;
    const int r = record(pred, rec ? i - d : 0, rec ? kk : 0, rec ? jj : 0, KD, chunks);
    const int act = rec ? r : kActR;
    const int a0 = lane_int(act, 0);
    const int a1 = lane_int(act, 1 + a0);
    const int a2 = lane_int(act, 4 + 3 * a0 + a1);
    const int a3 = lane_int(act, 13 + 9 * a0 + 3 * a1 + a2);
    const int mine = lane == 0 ? a0 : lane == 1 ? a1 : lane == 2 ? a2 : a3;
    if (lane < kLookUnits && i - lane >= 0) a.action[i - lane] = (uint8_t)mine;
    const int acts[4] = {a0, a1, a2, a3};
#pragma unroll
    for (int m = 0; m < kLookUnits; ++m) {
      const int ubh = lane_int(bh, m), ubl = lane_int(bl, m), url = lane_int(rl, m);
      if (i - m >= 0) {
        if (acts[m] == kActH) j -= ubh;
        if (acts[m] == kActL) {
          j -= ubl;
          k -= url;
        }
      }
    }
    bh = nbh;
    bl = nbl;
    rl = nrl;
  }
}

__device__ __forceinline__ double lane_f64(double v, int lane) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), lane);
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// Memory and risk of the chosen actions, summed in unit order (one wave:
// the inputs of 64 units are loaded at once, one chunk ahead, and the
// additions stay sequential).  A unit whose action adds nothing adds +0.0,
// which leaves the sums unchanged: they start at +0.0 and every chosen cost
// is finite and non-negative, so neither sum is ever -0.0.
struct UnitTotals {
  double mem, risk;
};

__device__ __forceinline__ UnitTotals unit_costs(const AllocArgs &a, int u) {
  UnitTotals c{0.0, 0.0};
  if (u < a.U) {
    const int act = a.action[u];
    if (act == kActH) c.mem = a.dm_h[u];
    if (act == kActL) {
      c.mem = a.dm_l[u];
      c.risk = a.psi[u];
    }
  }
  return c;
}

__global__ __launch_bounds__(kWave) void totals_kernel(const AllocArgs a) {
  const int lane = (int)threadIdx.x;
  double mem = 0.0, risk = 0.0;
  UnitTotals c = unit_costs(a, lane);
  for (int base = 0; base < a.U; base += kWave) {
    const UnitTotals next = unit_costs(a, base + kWave + lane);
    // all 64 lanes, unrolled (constant lane indices): lanes past the last
    // unit hold +0.0, which leaves the sums unchanged
#pragma unroll
    for (int t = 0; t < kWave; ++t) {
      mem += lane_f64(c.mem, t);
      risk += lane_f64(c.risk, t);
    }
    c = next;
  }
  if (lane == 0) {
    a.totals[1] = mem;
    a.totals[2] = risk;
  }
}

}  // namespace

AllocLayout alloc_layout(int U, int KB, int KD) {
  auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
  AllocLayout l{};
  l.S = (KB + kWave - 1) / kWave * kWave;
  l.cells = (int64_t)l.S * KD;
  l.off_costs = 0;
  l.off_f0 = up(sizeof(AllocUnitCost) * (size_t)(U > 0 ? U : 1));
  l.off_f1 = l.off_f0 + up(sizeof(double) * (size_t)l.cells);
  l.off_partial = l.off_f1 + up(sizeof(double) * (size_t)l.cells);
  l.off_pred = l.off_partial + up(sizeof(Best) * kPartials);
  l.pred_bytes_per_unit = (size_t)(l.cells / kWave) * 16;
  l.bytes = l.off_pred + up(l.pred_bytes_per_unit * (size_t)U);
  return l;
}

hipError_t launch_allocate(const AllocArgs &a, int KB, int KD, void *workspace, hipStream_t s) {
  const AllocLayout l = alloc_layout(a.U, KB, KD);
  char *ws = static_cast<char *>(workspace);
  AllocUnitCost *uc = reinterpret_cast<AllocUnitCost *>(ws + l.off_costs);
  double *f[2] = {reinterpret_cast<double *>(ws + l.off_f0),
                  reinterpret_cast<double *>(ws + l.off_f1)};
  Best *partial = reinterpret_cast<Best *>(ws + l.off_partial);
  uint64_t *pred = reinterpret_cast<uint64_t *>(ws + l.off_pred);

  if (a.U > 0) {
    hipLaunchKernelGGL(costs_kernel, dim3((a.U + 255) / 256), dim3(256), 0, s, a, uc);
    hipLaunchKernelGGL(reach_kernel, dim3(1), dim3(kReachThreads), 0, s, uc, a.U, KB);
  }
  const int grid = (int)((l.cells + kDpThreads - 1) / kDpThreads);
  hipLaunchKernelGGL(init_kernel, dim3(grid), dim3(kDpThreads), 0, s, f[0], f[1], l.cells);
  auto pred_of = [&](int i) {
    return reinterpret_cast<uint64_t *>(reinterpret_cast<char *>(pred) +
                                        l.pred_bytes_per_unit * (size_t)i);
  };
  // units in groups of kDpGroup (one launch each), the rest in a smaller
  // group; the table after launch t lives in f[t & 1]
  const size_t words = l.pred_bytes_per_unit / sizeof(uint64_t);
  int t = 0;
  for (int i = 0; i < a.U; i += kDpGroup, ++t) {
    const int g = a.U - i < kDpGroup ? a.U - i : kDpGroup;
    const dim3 gd(grid), bd(kDpThreads);
    double *src = f[t & 1], *dst = f[(t + 1) & 1];
    uint64_t *pr = pred_of(i);
    switch (g) {
      case 1: hipLaunchKernelGGL(dpn_kernel<1>, gd, bd, 0, s, src, dst, pr, words, uc + i, KB, KD, l.S); break;
      case 2: hipLaunchKernelGGL(dpn_kernel<2>, gd, bd, 0, s, src, dst, pr, words, uc + i, KB, KD, l.S); break;
      case 3: hipLaunchKernelGGL(dpn_kernel<3>, gd, bd, 0, s, src, dst, pr, words, uc + i, KB, KD, l.S); break;
      default: hipLaunchKernelGGL(dpn_kernel<4>, gd, bd, 0, s, src, dst, pr, words, uc + i, KB, KD, l.S); break;
    }
  }
  const int n_partial = grid < kPartials ? grid : kPartials;
  hipLaunchKernelGGL(terminal_partial_kernel, dim3(n_partial), dim3(kDpThreads), 0, s,
                     f[t & 1], l.cells, partial);
  hipLaunchKernelGGL(terminal_backtrack_kernel, dim3(1), dim3(kFinalThreads), 0, s, a, partial,
                     n_partial, pred, uc, l.S, KD);
  hipLaunchKernelGGL(totals_kernel, dim3(1), dim3(kWave), 0, s, a);
  return hipGetLastError();
}

}  // namespace hilore
