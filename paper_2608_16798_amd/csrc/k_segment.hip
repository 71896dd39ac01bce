// Policy-token compaction, rollout segmentation and group-relative advantages.
//
// Compaction keeps the positions t with M_t = 1 (Sec. 2.3.1: only valid policy-generated
// tokens are optimised) inside rollouts that are not excluded (Sec. 3.4: sandbox
// failures leave advantage estimation and policy optimisation), in ascending order.  Every
// later GEMM operand is gathered through this list, so masked tokens cost no MFMA work.
// Optionally (zero_grad: the caller's loss has no term but the advantage-weighted surrogate) the
// tokens of rollouts whose advantage is exactly 0 (an all-equal group, Sec. 2.3.2) go after all
// others, in their own ascending run: their surrogate gradient is exactly 0, so the backward
// covers only the first n_grad rows of the list while the forward covers all n_eff.
// The per-rollout count of kept tokens is the normaliser of the per-rollout token mean
// (masked GRPO objective, Sec. 2.3.2; shared-prefix tokens counted once, Sec. 3.2.3).
//
// Advantages follow the GRPO equation of Sec. 2.3.2 / Sec. 3.2.3: mean and population
// std over the non-excluded rollouts of a group (a task-harness pair, Sec. 3.3), with
// group keys treated as opaque and unordered.  All reductions run in a fixed order, in
// fp64, so results are bitwise reproducible.
#include "rlk_internal.h"

namespace rlk {

namespace {

constexpr int kThreads = 256;
constexpr int kPerThread = kScanTile / kThreads;  // 16 tokens per thread

__device__ inline int rollout_of(const int32_t* cu, int R, int64_t t) {
  // first r with cu[r+1] > t, clamped to [0, R-1]; tolerant of malformed cu
  int lo = 0, hi = R - 1;
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if ((int64_t)cu[mid + 1] > t) hi = mid; else lo = mid + 1;
  }
  return lo;
}

__device__ inline int wave_inclusive_scan(int v, int lane) {
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int n = __shfl_up(v, o, 64);
    if (lane >= o) v += n;
  }
  return v;
}

template <typename X>
__device__ inline X wave_sum(X v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__global__ void __launch_bounds__(kThreads) k_begin(WsHeader* hdr, const int32_t* cu, int R, int64_t N) {
  __shared__ int err;
  if (threadIdx.x == 0) err = 0;
  __syncthreads();
  int e = 0;
  if (R > 0) {
    for (int r = threadIdx.x; r < R; r += blockDim.x)
      if (cu[r] > cu[r + 1]) e |= RLK_DERR_CU_SEQLENS;
    if (threadIdx.x == 0 && (cu[0] != 0 || (int64_t)cu[R] != N)) e |= RLK_DERR_CU_SEQLENS;
  }
  if (e) atomicOr(&err, e);
  __syncthreads();
  if (threadIdx.x == 0) {
    hdr->status = err;
    hdr->n_eff = 0;
    hdr->n_grad = 0;
    hdr->n_groups = 0;
    hdr->n_valid = 0;
    hdr->ref_fallback = 0;
    hdr->n_dz_chunks = 0;
  }
}

__device__ inline bool keep_token(const uint8_t* mask, const int32_t* gid, int r, int64_t t) {
  bool k = mask ? (mask[t] != 0) : true;
  if (gid) k = k && (gid[r] >= 0);
  return k;
}

// keep[t]: 0 = not trained, 1 = trained, 2 = trained with an exactly zero surrogate gradient (its
// rollout's advantage is 0 and zero_adv is given).  blkcnt[b] counts the 1s of block b and
// blkcnt[nblk + b] its 2s, so one exclusive scan over both halves places every 2 after every 1.
__global__ void __launch_bounds__(kThreads)
k_count(const uint8_t* mask, const int32_t* cu, const int32_t* gid, const float* zero_adv, int R, int64_t N,
        uint8_t* keep, int32_t* blkcnt, int nblk) {
  __shared__ int partial[2][kThreads / 64];
  const int64_t t0 = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kPerThread;
  int cnt1 = 0, cnt2 = 0;
  if (t0 < N) {
    int r = rollout_of(cu, R, t0);
    for (int i = 0; i < kPerThread; ++i) {
      int64_t t = t0 + i;
      if (t >= N) break;
      while (r < R - 1 && (int64_t)cu[r + 1] <= t) ++r;
      const bool k = keep_token(mask, gid, r, t);
      const bool zg = k && zero_adv && zero_adv[r] == 0.0f;
      keep[t] = !k ? 0 : (zg ? 2 : 1);
      cnt1 += (k && !zg) ? 1 : 0;
      cnt2 += zg ? 1 : 0;
    }
  }
  cnt1 = wave_sum(cnt1);
  cnt2 = wave_sum(cnt2);
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (lane == 0) {
    partial[0][w] = cnt1;
    partial[1][w] = cnt2;
  }
  __syncthreads();
  if (threadIdx.x < 2) {
    int s = 0;
    for (int i = 0; i < kThreads / 64; ++i) s += partial[threadIdx.x][i];
    blkcnt[threadIdx.x * nblk + blockIdx.x] = s;
  }
}

// Exclusive scan of the per-block counts (both halves: nblk2 = 2 nblk); n_eff = the total, n_grad =
// the offset of the second half (the tokens with a gradient).  With a caller bound on the trained
// tokens (max_policy > 0) a larger total is flagged and both counts clamped to the bound, so every
// later kernel stays within the chunk loop the host sized for it.
__global__ void __launch_bounds__(1024) k_scan(const int32_t* blkcnt, int32_t* blkoff, int nblk2, int nblk,
                                               int32_t max_policy, WsHeader* hdr) {
  __shared__ int wsum[16];
  __shared__ int carry_s, ngrad_s;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  if (threadIdx.x == 0) carry_s = 0;
  __syncthreads();
  for (int base = 0; base < nblk2; base += 1024) {
    int i = base + threadIdx.x;
    int v = i < nblk2 ? blkcnt[i] : 0;
    int inc = wave_inclusive_scan(v, lane);
    if (lane == 63) wsum[w] = inc;
    __syncthreads();
    int woff = 0;
    for (int j = 0; j < w; ++j) woff += wsum[j];
    int carry = carry_s;
    if (i < nblk2) blkoff[i] = carry + woff + inc - v;
    if (i == nblk) ngrad_s = carry + woff + inc - v;
    __syncthreads();
    if (threadIdx.x == 1023) carry_s = carry + woff + inc;
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    int n = carry_s, g = ngrad_s;
    if (max_policy > 0 && n > max_policy) {
      atomicOr(&hdr->status, RLK_DERR_POLICY_BOUND);
      n = max_policy;
      g = g < n ? g : n;
    }
    hdr->n_eff = n;
    hdr->n_grad = g;
  }
}

__global__ void __launch_bounds__(kThreads)
k_write_idx(const uint8_t* keep, const int32_t* cu, int R, int64_t N, const int32_t* blkoff, int nblk,
            const int32_t* targets, int V, int32_t* idx, int32_t* tokr, int32_t* ytgt, float* zy,
            WsHeader* hdr) {
  __shared__ int wsum[2][kThreads / 64];
  const int64_t t0 = (int64_t)blockIdx.x * kScanTile + (int64_t)threadIdx.x * kPerThread;
  int cnt1 = 0, cnt2 = 0;
  for (int i = 0; i < kPerThread; ++i) {
    int64_t t = t0 + i;
    if (t < N) {
      cnt1 += keep[t] == 1;
      cnt2 += keep[t] == 2;
    }
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int inc1 = wave_inclusive_scan(cnt1, lane), inc2 = wave_inclusive_scan(cnt2, lane);
  if (lane == 63) {
    wsum[0][w] = inc1;
    wsum[1][w] = inc2;
  }
  __syncthreads();
  int off1 = blkoff[blockIdx.x], off2 = blkoff[nblk + blockIdx.x];
  for (int j = 0; j < w; ++j) {
    off1 += wsum[0][j];
    off2 += wsum[1][j];
  }
  off1 += inc1 - cnt1;
  off2 += inc2 - cnt2;
  if (cnt1 + cnt2 == 0) return;
  int r = rollout_of(cu, R, t0);
  int bad = 0;
  for (int i = 0; i < kPerThread; ++i) {
    int64_t t = t0 + i;
    if (t >= N) break;
    while (r < R - 1 && (int64_t)cu[r + 1] <= t) ++r;
    const uint8_t k = keep[t];
    if (k) {
      const int y = targets ? targets[t] : 0;
      if (y < 0 || y >= V) bad = 1;
      const int off = k == 1 ? off1++ : off2++;
      idx[off] = (int32_t)t;
      tokr[off] = r;
      ytgt[off] = y;
      zy[off] = 0.0f;
    }
  }
  if (bad) atomicOr(&hdr->status, RLK_DERR_TARGET);
}

__device__ inline int lower_bound_i32(const int32_t* a, int n, int64_t key) {
  int lo = 0, hi = n;
  while (lo < hi) {
    int mid = (lo + hi) >> 1;
    if ((int64_t)a[mid] < key) lo = mid + 1; else hi = mid;
  }
  return lo;
}

__global__ void __launch_bounds__(kThreads)
k_rollout_offsets(const int32_t* cu, int R, int64_t N, const int32_t* idx, const float* zero_adv,
                  const WsHeader* hdr, int32_t* rstart, int32_t* rnpol) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= R) return;
  // the rollout's tokens form one ascending run inside its part of the list: [0, n_grad) or, for a
  // rollout of zero advantage, [n_grad, n_eff)
  const int ng = hdr->n_grad, n = hdr->n_eff;
  const bool second = zero_adv && zero_adv[r] == 0.0f;
  const int lo = second ? ng : 0, hi = second ? n : ng;
  int64_t a = cu[r], b = cu[r + 1];
  a = a < 0 ? 0 : (a > N ? N : a);
  b = b < a ? a : (b > N ? N : b);
  int s = lo + lower_bound_i32(idx + lo, hi - lo, a);
  int e = lo + lower_bound_i32(idx + lo, hi - lo, b);
  rstart[r] = s;
  rnpol[r] = e - s;
}

// ---- group-relative advantages ----
//
// Segmentation by sorting: the (key, rollout) pairs of the non-excluded rollouts are sorted in one
// workgroup (bitonic network in LDS, R <= kMaxRollouts), so each group becomes a run of consecutive
// entries with its members in ascending rollout order; a scan over the run starts gives the dense
// group index (the rank of the key among the sorted distinct keys).  The statistics are then a
// segmented reduction: one wavefront per run.  O(R log^2 R) work for the sort, O(R) for the rest.

constexpr int kSortThreads = 1024;
constexpr int kSortMax = 16384;  // = kMaxRollouts: 128 KiB of 64-bit sort entries in LDS
static_assert(kSortMax >= kMaxRollouts, "sort capacity");

// entry = (key' << 32) | rollout with key' = key for a kept rollout and 0xFFFFFFFF for an excluded one
// (and for the padding), so kept rollouts sort first, by key, then by rollout.
__device__ inline uint64_t sort_entry(const int32_t* gid, int R, int i) {
  if (i >= R) return ~0ull;
  const int32_t key = gid[i];
  const uint32_t hi = key >= 0 ? (uint32_t)key : 0xFFFFFFFFu;
  return ((uint64_t)hi << 32) | (uint32_t)i;
}

__global__ void __launch_bounds__(kSortThreads)
k_group_sort(const int32_t* gid, int R, int32_t* members, int32_t* gstart, int32_t* gidx, WsHeader* hdr) {
  __shared__ uint64_t e[kSortMax];
  __shared__ int wsum[kSortThreads / 64];
  __shared__ int carry_s;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  int P = 1;
  while (P < R) P <<= 1;
  for (int i = tid; i < P; i += kSortThreads) e[i] = sort_entry(gid, R, i);
  __syncthreads();
  // bitonic sort of P entries, ascending
  for (int k = 2; k <= P; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      for (int i = tid; i < P; i += kSortThreads) {
        const int l = i ^ j;
        if (l > i) {
          const uint64_t a = e[i], b = e[l];
          const bool up = (i & k) == 0;
          if ((a > b) == up) {
            e[i] = b;
            e[l] = a;
          }
        }
      }
      __syncthreads();
    }
  }
  // kept entries come first; a run starts where the key differs from the previous entry's
  if (tid == 0) carry_s = 0;
  __syncthreads();
  for (int base = 0; base < R; base += kSortThreads) {
    const int i = base + tid;
    const uint64_t v = i < R ? e[i] : ~0ull;
    const bool kept = (v >> 32) != 0xFFFFFFFFull;
    const int start = kept && (i == 0 || (e[i - 1] >> 32) != (v >> 32)) ? 1 : 0;
    const int inc = wave_inclusive_scan(start, lane);
    if (lane == 63) wsum[w] = inc;
    __syncthreads();
    int off = carry_s;
    for (int j = 0; j < w; ++j) off += wsum[j];
    const int q = off + inc - 1;  // dense index of this entry's group
    if (kept) {
      const int r = (int)(uint32_t)v;
      members[i] = r;
      gidx[r] = q;
      if (start) gstart[q] = i;
    } else if (i < R) {
      gidx[(int)(uint32_t)v] = -1;
    }
    __syncthreads();
    if (tid == kSortThreads - 1) carry_s = off + inc;
    __syncthreads();
  }
  // n_valid = number of kept entries: the first excluded (or padding) position
  if (tid == 0) {
    int lo = 0, hi = R;
    while (lo < hi) {
      const int mid = (lo + hi) >> 1;
      if ((e[mid] >> 32) != 0xFFFFFFFFull) lo = mid + 1; else hi = mid;
    }
    gstart[carry_s] = lo;  // end of the last run
    hdr->n_groups = carry_s;
    hdr->n_valid = lo;
  }
}

// Segmented statistics: one wavefront per group over its members (ascending rollout order), lanes
// striding the run, partial sums combined by a fixed shuffle tree: mean and population std in
// fp64, and whether every reward of the group is bitwise equal.
__global__ void __launch_bounds__(kThreads)
k_group_stats(const float* rewards, const int32_t* members, const int32_t* gstart, const WsHeader* hdr,
              int32_t* gsize, double* gmu, double* gsig, int32_t* geq) {
  const int lane = threadIdx.x & 63;
  const int q = blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
  if (q >= hdr->n_groups) return;
  const int b = gstart[q], n = gstart[q + 1] - b;
  double sum = 0.0;
  float mn = INFINITY, mx = -INFINITY;
  for (int i = lane; i < n; i += 64) {
    const float v = rewards[members[b + i]];
    sum += (double)v;
    mn = fminf(mn, v);
    mx = fmaxf(mx, v);
  }
  sum = wave_sum(sum);
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    mn = fminf(mn, __shfl_xor(mn, o, 64));
    mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  }
  const double mu = n > 0 ? sum / (double)n : 0.0;
  double ss = 0.0;
  for (int i = lane; i < n; i += 64) {
    const double dv = (double)rewards[members[b + i]] - mu;
    ss += dv * dv;
  }
  ss = wave_sum(ss);
  if (lane == 0) {
    gsize[q] = n;
    gmu[q] = mu;
    gsig[q] = n > 0 ? sqrt(ss / (double)n) : 0.0;
    geq[q] = (mn == mx) ? 1 : 0;
  }
}

__global__ void __launch_bounds__(kThreads)
k_advantage(const float* rewards, const int32_t* gidx, int R, const double* gmu, const double* gsig,
            const int32_t* geq, float adv_eps, float* adv) {
  const int r = blockIdx.x * blockDim.x + threadIdx.x;
  if (r >= R) return;
  const int q = gidx[r];
  double a = 0.0;
  if (q >= 0 && !geq[q]) a = ((double)rewards[r] - gmu[q]) / (gsig[q] + (double)adv_eps);
  adv[r] = (float)a;
}

inline dim3 blocks_for(int64_t n, int per) { return dim3((unsigned)((n + per - 1) / per)); }

}  // namespace

hipError_t launch_begin(int32_t* status_hdr, const int32_t* cu, int R, int64_t N, hipStream_t s) {
  prof_mark(KK_BEGIN, true, s);
  k_begin<<<1, kThreads, 0, s>>>(reinterpret_cast<WsHeader*>(status_hdr), cu, R, N);
  prof_mark(KK_BEGIN, false, s);
  return hipGetLastError();
}

hipError_t launch_compact(const uint8_t* mask, const int32_t* cu, const int32_t* gid, int R, int64_t N,
                          const int32_t* targets, int V, int32_t max_policy, const float* zero_adv, char* ws,
                          const WsLayout& L, hipStream_t s) {
  WsHeader* hdr = reinterpret_cast<WsHeader*>(ws + L.hdr);
  uint8_t* keep = reinterpret_cast<uint8_t*>(ws + L.keep);
  int32_t* blkcnt = reinterpret_cast<int32_t*>(ws + L.blkcnt);
  int32_t* blkoff = reinterpret_cast<int32_t*>(ws + L.blkoff);
  if (N > 0) {
    prof_mark(KK_COUNT, true, s);
    k_count<<<L.nblk, kThreads, 0, s>>>(mask, cu, gid, zero_adv, R, N, keep, blkcnt, L.nblk);
    prof_mark(KK_COUNT, false, s);
    prof_mark(KK_SCAN, true, s);
    k_scan<<<1, 1024, 0, s>>>(blkcnt, blkoff, 2 * L.nblk, L.nblk, max_policy, hdr);
    prof_mark(KK_SCAN, false, s);
    prof_mark(KK_WRITE_IDX, true, s);
    k_write_idx<<<L.nblk, kThreads, 0, s>>>(keep, cu, R, N, blkoff, L.nblk, targets, V,
                                             reinterpret_cast<int32_t*>(ws + L.idx),
                                             reinterpret_cast<int32_t*>(ws + L.tokr),
                                             reinterpret_cast<int32_t*>(ws + L.ytgt),
                                             reinterpret_cast<float*>(ws + L.zy), hdr);
    prof_mark(KK_WRITE_IDX, false, s);
  }
  if (R > 0) {
    prof_mark(KK_ROLLOUT_OFFSETS, true, s);
    k_rollout_offsets<<<blocks_for(R, kThreads), kThreads, 0, s>>>(
        cu, R, N, reinterpret_cast<const int32_t*>(ws + L.idx), zero_adv, hdr,
        reinterpret_cast<int32_t*>(ws + L.rstart), reinterpret_cast<int32_t*>(ws + L.rnpol));
    prof_mark(KK_ROLLOUT_OFFSETS, false, s);
  }
  return hipGetLastError();
}

hipError_t launch_advantage(int R, const float* rewards, const int32_t* gid, float adv_eps, int32_t* members,
                            int32_t* gstart, int32_t* gidx, int32_t* gsize, double* gmu, double* gsig, int32_t* geq,
                            float* adv, WsHeader* hdr, hipStream_t s) {
  if (R <= 0) return hipSuccess;
  if (R > kSortMax) return hipErrorInvalidValue;
  prof_mark(KK_GROUP_RANK, true, s);
  k_group_sort<<<1, kSortThreads, 0, s>>>(gid, R, members, gstart, gidx, hdr);
  prof_mark(KK_GROUP_RANK, false, s);
  prof_mark(KK_GROUP_STATS, true, s);
  k_group_stats<<<blocks_for(R, kThreads / 64), kThreads, 0, s>>>(rewards, members, gstart, hdr, gsize, gmu, gsig,
                                                                   geq);
  prof_mark(KK_GROUP_STATS, false, s);
  prof_mark(KK_ADVANTAGE, true, s);
  k_advantage<<<blocks_for(R, kThreads), kThreads, 0, s>>>(rewards, gidx, R, gmu, gsig, geq, adv_eps, adv);
  prof_mark(KK_ADVANTAGE, false, s);
  return hipGetLastError();
}

}  // namespace rlk
