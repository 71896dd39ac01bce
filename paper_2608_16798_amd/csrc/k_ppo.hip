// PPO path kernels (ClawGym II, Sec. 2.3.1 GAE and value loss; Sec. 3.2.3 simplified variant):
// masked generalised advantage estimation as a per-rollout reverse scan, and the masked
// mean-squared value loss with its gradient.
//
// GAE over a rollout's policy rows t_1 < ... < t_n (tool rows are stepped over):
//   delta_j = gamma V[t_{j+1}] - V[t_j]  (j < n),   delta_n = R - V[t_n],
//   A_j = delta_j + c A_{j+1}, c = gamma lambda,  returns = A + V.
// One workgroup per rollout walks the rollout backwards in chunks of 256 rows.  Thread i of a
// chunk holds row e - 1 - i, so increasing thread order is decreasing row order and both
// quantities are inclusive scans over threads, carried from chunk to chunk:
//   - the value of the nearest later policy row (a "latest seen" scan), which gives delta;
//   - A as the composition of the affine maps x -> (policy ? c x + delta : x).
#include "rlk_internal.h"

namespace rlk {

namespace {

constexpr int kGaeThreads = 256;

__device__ __forceinline__ int64_t clamp64(int64_t v, int64_t lo, int64_t hi) { return v < lo ? lo : (v > hi ? hi : v); }

__global__ void __launch_bounds__(kGaeThreads)
k_gae(int64_t N, const int32_t* cu, const uint8_t* mask, const float* values, const float* rewards,
      const int32_t* gid, float gamma, float lam, float* adv, float* ret) {
  __shared__ int s_has[kGaeThreads];
  __shared__ double s_val[kGaeThreads];
  __shared__ double s_a[kGaeThreads], s_b[kGaeThreads];
  const int r = blockIdx.x;
  const int i = threadIdx.x;
  const int64_t s0 = clamp64(cu[r], 0, N), s1 = clamp64(cu[r + 1], s0, N);
  const bool excluded = gid && gid[r] < 0;
  const double c = (double)gamma * (double)lam;
  const double R = (double)rewards[r];
  int carry_has = 0;        // a policy row exists after the current chunk
  double carry_val = 0.0;   // its value
  double carry_A = 0.0;     // advantage of the nearest policy row at or after the chunk's end
  for (int64_t e = s1; e > s0; e -= kGaeThreads) {
    const int64_t t = e - 1 - i;
    const bool in = t >= s0;
    const bool pol = in && !excluded && mask[t] != 0;
    const double v = pol ? (double)values[t] : 0.0;
    // (1) nearest later policy row: exclusive "latest seen" scan over threads
    s_has[i] = pol;
    s_val[i] = v;
    __syncthreads();
    for (int off = 1; off < kGaeThreads; off <<= 1) {
      int h = 0;
      double x = 0.0;
      const bool take = i >= off && !s_has[i];
      if (take) {
        h = s_has[i - off];
        x = s_val[i - off];
      }
      __syncthreads();
      if (take) {
        s_has[i] = h;
        s_val[i] = x;
      }
      __syncthreads();
    }
    int nh = carry_has;
    double nv = carry_val;
    if (i > 0 && s_has[i - 1]) {
      nh = 1;
      nv = s_val[i - 1];
    }
    const double delta = pol ? ((nh ? (double)gamma * nv : R) - v) : 0.0;
    const int last_has = s_has[kGaeThreads - 1];
    const double last_val = s_val[kGaeThreads - 1];
    __syncthreads();
    // (2) A: inclusive scan of the affine maps x -> a x + b over threads (thread 0 applied first)
    double a = pol ? c : 1.0, b = pol ? delta : 0.0;
    s_a[i] = a;
    s_b[i] = b;
    __syncthreads();
    for (int off = 1; off < kGaeThreads; off <<= 1) {
      double pa = 1.0, pb = 0.0;
      if (i >= off) {
        pa = s_a[i - off];
        pb = s_b[i - off];
      }
      __syncthreads();
      if (i >= off) {
        // this map after the earlier one: x -> a (pa x + pb) + b
        b = a * pb + b;
        a = a * pa;
        s_a[i] = a;
        s_b[i] = b;
      }
      __syncthreads();
    }
    const double A = a * carry_A + b;
    if (in) {
      adv[t] = pol ? (float)A : 0.0f;
      if (ret) ret[t] = pol ? (float)(A + v) : 0.0f;
    }
    const double chunk_a = s_a[kGaeThreads - 1], chunk_b = s_b[kGaeThreads - 1];
    __syncthreads();
    carry_A = chunk_a * carry_A + chunk_b;
    if (last_has) {
      carry_has = 1;
      carry_val = last_val;
    }
  }
}

// ---- value loss: per-rollout fp64 partial sums, one block for the totals, then the gradient.
__global__ void __launch_bounds__(256)
k_value_partial(int64_t N, const int32_t* cu, const uint8_t* mask, const float* values, const float* ret,
                const int32_t* gid, double* part) {
  __shared__ double sh[4][2];
  const int r = blockIdx.x;
  const int64_t s0 = clamp64(cu[r], 0, N), s1 = clamp64(cu[r + 1], s0, N);
  double ss = 0.0, cnt = 0.0;
  if (!(gid && gid[r] < 0)) {
    for (int64_t t = s0 + threadIdx.x; t < s1; t += 256) {
      if (!mask[t]) continue;
      const double d = (double)values[t] - (double)ret[t];
      ss += d * d;
      cnt += 1.0;
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    ss += __shfl_xor(ss, o, 64);
    cnt += __shfl_xor(cnt, o, 64);
  }
  if ((threadIdx.x & 63) == 0) {
    sh[threadIdx.x >> 6][0] = ss;
    sh[threadIdx.x >> 6][1] = cnt;
  }
  __syncthreads();
  if (threadIdx.x < 2) part[(int64_t)r * 2 + threadIdx.x] = sh[0][threadIdx.x] + sh[1][threadIdx.x] +
                                                             sh[2][threadIdx.x] + sh[3][threadIdx.x];
}

__global__ void __launch_bounds__(1024) k_value_final(int R, const double* part, double* total, float* loss) {
  __shared__ double sh[16][2];
  double ss = 0.0, cnt = 0.0;
  for (int r = threadIdx.x; r < R; r += 1024) {
    ss += part[(int64_t)r * 2];
    cnt += part[(int64_t)r * 2 + 1];
  }
  for (int o = 32; o > 0; o >>= 1) {
    ss += __shfl_xor(ss, o, 64);
    cnt += __shfl_xor(cnt, o, 64);
  }
  if ((threadIdx.x & 63) == 0) {
    sh[threadIdx.x >> 6][0] = ss;
    sh[threadIdx.x >> 6][1] = cnt;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    double a = 0.0, n = 0.0;
    for (int k = 0; k < 16; ++k) {
      a += sh[k][0];
      n += sh[k][1];
    }
    total[0] = n;
    loss[0] = n > 0 ? (float)(a / n) : 0.0f;
  }
}

__global__ void __launch_bounds__(256)
k_value_grad(int64_t N, const int32_t* cu, const uint8_t* mask, const float* values, const float* ret,
             const int32_t* gid, const double* total, float* dv) {
  const int r = blockIdx.x;
  const int64_t s0 = clamp64(cu[r], 0, N), s1 = clamp64(cu[r + 1], s0, N);
  const bool excluded = gid && gid[r] < 0;
  const double n = total[0];
  for (int64_t t = s0 + threadIdx.x; t < s1; t += 256) {
    const bool on = !excluded && mask[t] && n > 0;
    dv[t] = on ? (float)(2.0 * ((double)values[t] - (double)ret[t]) / n) : 0.0f;
  }
}

}  // namespace

hipError_t launch_gae(int64_t N, int R, const int32_t* cu, const uint8_t* mask, const float* values,
                      const float* rewards, const int32_t* gid, float gamma, float lam, float* adv, float* ret,
                      hipStream_t s) {
  prof_mark(KK_GAE, true, s);
  k_gae<<<R, kGaeThreads, 0, s>>>(N, cu, mask, values, rewards, gid, gamma, lam, adv, ret);
  prof_mark(KK_GAE, false, s);
  return hipGetLastError();
}

hipError_t launch_value_loss(int64_t N, int R, const int32_t* cu, const uint8_t* mask, const float* values,
                             const float* ret, const int32_t* gid, double* part, double* total, float* loss,
                             float* dv, hipStream_t s) {
  prof_mark(KK_VALUE_LOSS, true, s);
  k_value_partial<<<R, 256, 0, s>>>(N, cu, mask, values, ret, gid, part);
  k_value_final<<<1, 1024, 0, s>>>(R, part, total, loss);
  if (dv) k_value_grad<<<R, 256, 0, s>>>(N, cu, mask, values, ret, gid, total, dv);
  prof_mark(KK_VALUE_LOSS, false, s);
  return hipGetLastError();
}

}  // namespace rlk
