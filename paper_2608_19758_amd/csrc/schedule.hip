// Work plan of the sparse attention and the merge of its KV splits
// (Sec. 3.3 Eq. split and Eq. cost).
//
// plan_kernel runs once per call after the kept lists exist. The cost of a
// unit (sequence b, KV head h, query block I) is proportional to its number
// of 64-key steps (Eq. cost): two per kept block, one per 64 corrected
// blocks, plus a fixed per-item share. In the cost-balanced mode (splits ==
// 0) every unit whose cost exceeds a step budget S is cut into
// U = ceil(cost / S) parts (at most kMaxRowSplits), and S is chosen so that
// the whole call has about target_items items of at most S steps (never
// less than kMinSplitSteps, and large enough for the partial-output
// capacity of the workspace). A fixed count n >= 1 cuts every unit into n.
// Part u of a unit walks kept-list positions [u ceil(T/U), min((u+1)
// ceil(T/U), T)) of its T kept blocks and the u-th of U equal ranges of the
// pruned blocks (Eq. split). The plan is an item table in attention order
// (decreasing query block, heaviest first, units without queries left out),
// per-unit {U, first partial slot}, and the list of units with U > 1.
//
// combine_kernel merges the parts of every split unit with the log-sum-exp
// weights: M = max_u m_u, w_u = 2^(m_u - M), O = c_v sum_u w_u o_u /
// sum_u w_u l_u, LSE = (M + log2 sum_u w_u l_u - offset) ln 2. Parts that saw
// no key have m_u = -inf and weight 0. It is HBM-bound (U x 520 bytes read
// and 256 written per packed row) and persistent over (split unit, 8-row
// group) pairs.
#include <atomic>
#include <algorithm>

#include "kernels.h"

namespace fp2 {

namespace {

constexpr float kLn2 = 0.69314718055994530942f;
constexpr int kPlanThreads = 1024;
constexpr int kPlanWaves = kPlanThreads / 64;
constexpr int kMinSplitSteps = 16;   // smallest step budget of an item
constexpr int kItemSteps = 2;        // fixed per-item cost (query load, set-up), in steps
constexpr int kMaxRowSplits = 32;    // one part per lane of the combine's half-wave
constexpr int kCostCache = 16384;    // units whose costs the plan keeps in LDS (64 KiB)

__device__ double block_sum(double v, double* sh) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  __syncthreads();
  if (lane == 0) sh[w] = v;
  __syncthreads();
  double t = 0.0;
  for (int k = 0; k < kPlanWaves; ++k) t += sh[k];
  return t;
}

__device__ int block_max(int v, int* sh) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
  __syncthreads();
  if (lane == 0) sh[w] = v;
  __syncthreads();
  int t = sh[0];
  for (int k = 1; k < kPlanWaves; ++k) t = max(t, sh[k]);
  return t;
}

// Exclusive prefix sum over the workgroup (thread order); `total` is the sum
// over all threads.
__device__ int block_excl_scan(int v, int* sh, int& total) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  int inc = v;
  for (int o = 1; o < 64; o <<= 1) {
    const int t = __shfl_up(inc, o, 64);
    if (lane >= o) inc += t;
  }
  __syncthreads();
  if (lane == 63) sh[w] = inc;
  __syncthreads();
  int pre = 0;
  total = 0;
  for (int k = 0; k < kPlanWaves; ++k) {
    const int x = sh[k];
    pre += k < w ? x : 0;
    total += x;
  }
  return pre + inc - v;
}

// Walk over attention-order indices q = (nbmax - 1 - I) * nbh + bh from a
// start index: unit row (b * Hkv + h) * nbmax + I, sequence b and query
// block I, with one division at the start and none per step.
struct UnitWalk {
  int I, bh, b, h, nbh, hkv, nbmax;
  __device__ UnitWalk(const Problem& p, int q0) : nbh(p.batch * p.hkv), hkv(p.hkv), nbmax(p.nbmax) {
    I = nbmax - 1 - q0 / nbh;
    bh = q0 % nbh;
    b = bh / hkv;
    h = bh - b * hkv;
  }
  __device__ int row() const { return bh * nbmax + I; }
  __device__ void next() {
    ++bh;
    if (++h == hkv) {
      h = 0;
      ++b;
    }
    if (bh == nbh) {
      bh = b = h = 0;
      --I;
    }
  }
};

__global__ __launch_bounds__(kPlanThreads) void plan_kernel(Problem p, KeptLists kl, Plan plan,
                                                            int wpu) {
  __shared__ double shd[kPlanWaves];
  __shared__ int shi[kPlanWaves];
  __shared__ int sc[kCostCache];
  const int tid = threadIdx.x;
  const int nbh = p.batch * p.hkv;
  const int R = nbh * p.nbmax;
  // thread tid owns the attention-order indices q in [q0, q1): contiguous, so
  // one scan over the threads orders the whole table
  const int per = (R + kPlanThreads - 1) / kPlanThreads;
  const int q0 = min(R, tid * per), q1 = min(R, q0 + per);

  // cost in steps of one row slice of every unit with queries (-1: none),
  // kept in LDS when the table is small enough (indexed by q), else in
  // rowinfo.x until the plan overwrites it
  const bool in_lds = R <= kCostCache;
  auto cost_at = [&](int q, int row) -> int { return in_lds ? sc[q] : plan.rowinfo[row].x; };
  double tot = 0.0;
  int mx = 0;
  // eight units at a time: their loads are issued together
  UnitWalk u(p, q0);
  for (int qb = q0; qb < q1; qb += 8) {
    int row[8], I[8], b[8], cnt[8], lq[8], lk[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      row[j] = u.row();
      I[j] = u.I;
      b[j] = u.b;
      u.next();
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const bool v = qb + j < q1;
      cnt[j] = v ? kl.cnt[row[j]] : 0;
      lq[j] = v ? p.cu[b[j] + 1] - p.cu[b[j]] : 0;
      lk[j] = v ? p.cuk[b[j] + 1] - p.cuk[b[j]] : 0;
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      if (qb + j >= q1) break;
      const int Lq = lq[j];
      int cost = -1;
      if (I[j] * p.qtile < Lq) {
        const int Ia = (lk[j] - Lq + min(Lq, (I[j] + 1) * p.qtile) - 1) / kBlock;
        const int pruned = p.corr ? max(0, Ia + 1 - cnt[j]) : 0;   // at most, below the last block
        cost = 2 * cnt[j] + (pruned + 63) / 64 + kItemSteps;
        tot += (double)cost * wpu;
        mx = max(mx, cost);
      }
      if (in_lds)
        sc[qb + j] = cost;
      else
        plan.rowinfo[row[j]] = make_int2(cost, -1);
    }
  }
  tot = block_sum(tot, shd);   // (its barriers also publish sc)
  mx = block_max(mx, shi);

  // step budget of the cost-balanced mode
  int S = 0;
  if (p.splits == 0) {
    S = max(kMinSplitSteps, (int)ceil(tot / (double)max(1, plan.target_items)));
    while (S < mx) {   // grow S until the parts fit the partial-output slots
      int need = 0;
      UnitWalk w(p, q0);
      for (int q = q0; q < q1; ++q, w.next()) {
        const int cost = cost_at(q, w.row());
        if (cost > S) need += min(kMaxRowSplits, (cost + S - 1) / S);
      }
      need = (int)block_sum((double)need, shd);
      if (need <= plan.cap_slots) break;
      S *= 2;
    }
  }
  auto parts = [&](int cost) -> int {
    if (cost < 0) return 0;
    if (p.splits > 0) return p.splits;
    return cost > S ? min(kMaxRowSplits, (cost + S - 1) / S) : 1;
  };

  // items in attention order, partial slots and split units: this thread's
  // totals, their exclusive scans over the threads, then the entries
  int ni = 0, ns = 0, nsr = 0;
  {
    UnitWalk w(p, q0);
    for (int q = q0; q < q1; ++q, w.next()) {
      const int U = parts(cost_at(q, w.row()));
      ni += U * wpu;
      ns += U > 1 ? U : 0;
      nsr += U > 1 ? 1 : 0;
    }
  }
  int ti, ts, tsr;
  int bi = block_excl_scan(ni, shi, ti);
  int bs = block_excl_scan(ns, shi, ts);
  int bsr = block_excl_scan(nsr, shi, tsr);
  UnitWalk w(p, q0);
  for (int q = q0; q < q1; ++q, w.next()) {
    const int row = w.row();
    const int U = parts(cost_at(q, row));
    if (U == 0) {
      if (in_lds) plan.rowinfo[row] = make_int2(-1, -1);
      continue;
    }
    const int slot = U > 1 ? bs : -1;
    plan.rowinfo[row] = make_int2(U, slot);
    if (U > 1) {
      plan.splitrows[bsr++] = row;
      bs += U;
    }
    for (int k = 0; k < U * wpu; ++k) plan.items[bi + k] = make_int4(q, k, U, slot);
    bi += U * wpu;
  }
  if (tid == 0) {
    plan.counts[0] = 0;
    plan.counts[1] = ti;
    plan.counts[2] = tsr;
  }
}

template <int FP8>
__global__ __launch_bounds__(256) void combine_kernel(Problem p, Plan plan,
                                                      uint16_t* __restrict__ out,
                                                      float* __restrict__ lse) {
  const int G = p.g, rpu = G * p.qtile, groups = rpu / 8;
  const int work = plan.counts[2] * groups;
  const int lane = threadIdx.x & 31, sub = threadIdx.x >> 5;
  const int c = lane * 4;
  const float off = FP8 ? 8.f : 0.f;
#pragma unroll 1
  for (int wk = blockIdx.x; wk < work; wk += gridDim.x) {
    const int sr = wk / groups, grp = wk - sr * groups;
    const int row = plan.splitrows[sr];
    const int2 ri = plan.rowinfo[row];
    const int U = ri.x, slot0 = ri.y;
    const int I = row % p.nbmax, bh = row / p.nbmax;
    const int b = bh / p.hkv, h = bh % p.hkv;
    const int pr = grp * 8 + sub;              // packed row of this half-wave
    const int pos = I * p.qtile + pr / G;
    if (pos >= p.cu[b + 1] - p.cu[b]) continue;
    // lane u < U holds part u's {m, l}
    float m = -INFINITY, l = 0.f;
    if (lane < U) {
      const float2 ml = *(const float2*)(plan.part_ml + 2 * ((int64_t)(slot0 + lane) * rpu + pr));
      m = ml.x;
      l = ml.y;
    }
    float M = m;
    for (int o = 16; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o, 32));
    const float wgt = m == -INFINITY ? 0.f : fast_exp2(m - M);
    float lt = wgt * l;
    for (int o = 16; o > 0; o >>= 1) lt += __shfl_xor(lt, o, 32);
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int u0 = 0; u0 < U; u0 += 4) {   // four parts' loads in flight at a time
      float wu[4];
      float4 o[4];
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int u = u0 + k;
        wu[k] = __shfl(wgt, u & 31, 32);
        o[k] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (u < U && wu[k] != 0.f)
          o[k] = *(const float4*)(plan.part_o + ((int64_t)(slot0 + u) * rpu + pr) * kHeadDim + c);
        else
          wu[k] = 0.f;
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        acc.x = fmaf(wu[k], o[k].x, acc.x);
        acc.y = fmaf(wu[k], o[k].y, acc.y);
        acc.z = fmaf(wu[k], o[k].z, acc.z);
        acc.w = fmaf(wu[k], o[k].w, acc.w);
      }
    }
    const float inv = (FP8 ? p.v_scale[h] : 1.f) / lt;
    const int hq = h * G + pr % G;
    const int64_t t = (int64_t)p.cu[b] + pos;
    uint2 v;
    v.x = pack_bf16x2(acc.x * inv, acc.y * inv);
    v.y = pack_bf16x2(acc.z * inv, acc.w * inv);
    *(uint2*)(out + (t * p.hq + hq) * kHeadDim + c) = v;
    if (lse && lane == 0) lse[t * p.hq + hq] = (M + fast_log2(lt) - off) * kLn2;
  }
}

}  // namespace

// Compute units of the current device, queried once per device; the cache is
// atomic so that calls from several host threads are well defined (each may
// query and store the same value).
int device_compute_units() {
  static std::atomic<int> cus[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int n = cus[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
    cus[dev].store(n, std::memory_order_relaxed);
  }
  return n;
}

hipError_t launch_plan(const Problem& p, const KeptLists& kl, const Plan& plan, hipStream_t s) {
  if (p.batch == 0 || p.nbmax == 0) return hipSuccess;
  plan_kernel<<<1, kPlanThreads, 0, s>>>(p, kl, plan, attend_items_per_unit(p.g, p.qtile));
  return hipGetLastError();
}

hipError_t launch_combine(const Problem& p, const Plan& plan, void* out, float* lse,
                          hipStream_t s) {
  if (p.batch == 0 || p.nbmax == 0 || plan.cap_slots == 0) return hipSuccess;
  const int64_t bound = (int64_t)(plan.cap_slots / 2) * (p.g * p.qtile / 8);
  const unsigned grid = (unsigned)std::max<int64_t>(1, std::min<int64_t>(bound, 1024));
  if (p.fp8)
    combine_kernel<1><<<grid, 256, 0, s>>>(p, plan, (uint16_t*)out, lse);
  else
    combine_kernel<0><<<grid, 256, 0, s>>>(p, plan, (uint16_t*)out, lse);
  return hipGetLastError();
}

}  // namespace fp2
