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

// ---- linear value head V_t = w . h_t + b on the kept rows (mask = 1, rollout not excluded) and
// its backward.  Reductions run in a fixed order (wavefront trees, block partials in row order),
// so results are bitwise reproducible.
__device__ __forceinline__ int rollout_of_row(const int32_t* cu, int R, int64_t t) {
  int lo = 0, hi = R - 1;  // first r with cu[r+1] > t, clamped to [0, R-1]
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if ((int64_t)cu[mid + 1] > t) hi = mid; else lo = mid + 1;
  }
  return lo;
}

__device__ __forceinline__ bool kept_row(const uint8_t* mask, const int32_t* cu, const int32_t* gid, int R,
                                         int64_t t) {
  if (mask && !mask[t]) return false;
  return !gid || gid[rollout_of_row(cu, R, t)] >= 0;
}

template <typename T>
__device__ __forceinline__ void unpack8(const u32x4 v, float (&f)[16 / sizeof(T)]);
template <>
__device__ __forceinline__ void unpack8<bf16_t>(const u32x4 v, float (&f)[8]) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}
template <>
__device__ __forceinline__ void unpack8<float>(const u32x4 v, float (&f)[4]) {
  f[0] = __uint_as_float(v.x);
  f[1] = __uint_as_float(v.y);
  f[2] = __uint_as_float(v.z);
  f[3] = __uint_as_float(v.w);
}
__device__ __forceinline__ uint32_t bf16_pair(float lo, float hi) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (__bf16)lo) | ((uint32_t)__builtin_bit_cast(uint16_t, (__bf16)hi) << 16);
}

constexpr int kHeadRows = 256;    // rows per workgroup of the dW partial sums

// one wavefront per row
template <typename T>
__global__ void __launch_bounds__(256)
k_value_head_fwd(int64_t N, int d, const T* h, const T* w, float b, const uint8_t* mask, const int32_t* cu,
                 const int32_t* gid, int R, float* values) {
  constexpr int EPC = 16 / sizeof(T);
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= N) return;
  if (!kept_row(mask, cu, gid, R, t)) {
    if (lane == 0) values[t] = 0.0f;
    return;
  }
  const T* row = h + t * d;
  float acc = 0.0f;
  for (int c = lane; c < d / EPC; c += 64) {
    float x[EPC], y[EPC];
    unpack8<T>(*reinterpret_cast<const u32x4*>(row + c * EPC), x);
    unpack8<T>(*reinterpret_cast<const u32x4*>(w + c * EPC), y);
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc = fmaf(x[e], y[e], acc);
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
  if (lane == 0) values[t] = acc + b;
}

// dhidden rows: kept rows get (dh +) dV_t w, the others are zeroed unless accumulating
template <typename T>
__global__ void __launch_bounds__(256)
k_value_head_dh(int64_t N, int d, const T* w, const float* dv, const uint8_t* mask, const int32_t* cu,
                const int32_t* gid, int R, T* dh, int accumulate, float* gk) {
  constexpr int EPC = 16 / sizeof(T);
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= N) return;
  const bool keep = kept_row(mask, cu, gid, R, t);
  const float g = keep ? dv[t] : 0.0f;
  if (lane == 0) gk[t] = g;  // the row's gradient for the dw / db sums
  if (!dh || (!keep && accumulate)) return;
  T* row = dh + t * d;
  for (int c = lane; c < d / EPC; c += 64) {
    float y[EPC], o[EPC];
    unpack8<T>(*reinterpret_cast<const u32x4*>(w + c * EPC), y);
    if (accumulate) {
      unpack8<T>(*reinterpret_cast<const u32x4*>(row + c * EPC), o);
    } else {
#pragma unroll
      for (int e = 0; e < EPC; ++e) o[e] = 0.0f;
    }
#pragma unroll
    for (int e = 0; e < EPC; ++e) o[e] = fmaf(g, y[e], o[e]);
    u32x4 v;
    if constexpr (sizeof(T) == 2) {
      v = u32x4{bf16_pair(o[0], o[1]), bf16_pair(o[2], o[3]), bf16_pair(o[4], o[5]), bf16_pair(o[6], o[7])};
    } else {
      v = u32x4{__float_as_uint(o[0]), __float_as_uint(o[1]), __float_as_uint(o[2]), __float_as_uint(o[3])};
    }
    *reinterpret_cast<u32x4*>(row + c * EPC) = v;
  }
}

// dW partial sums over kHeadRows rows per workgroup: part[blk][j] = sum_t dV_t h_t[j] (fp32, row
// order), part_db[blk] = sum_t dV_t (fp64); each thread owns 16-byte column chunks.
template <typename T>
__global__ void __launch_bounds__(256)
k_value_head_dw_partial(int64_t N, int d, const T* h, const float* gk, float* part, double* part_db) {
  constexpr int EPC = 16 / sizeof(T);
  const int64_t t0 = (int64_t)blockIdx.x * kHeadRows, t1 = min(N, t0 + kHeadRows);
  for (int cb = 0; cb < d / EPC; cb += 256) {
    const int c = cb + threadIdx.x;
    float acc[EPC];
#pragma unroll
    for (int e = 0; e < EPC; ++e) acc[e] = 0.0f;
    double db = 0.0;
    // rows in groups of four: the row loads of a group are issued together (skipped for rows with
    // no gradient), then accumulated in row order
    for (int64_t t = t0; t < t1; t += 4) {
      float g4[4];
      u32x4 x4[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int64_t tt = t + u;
        g4[u] = 0.0f;
        x4[u] = u32x4{0, 0, 0, 0};
        if (tt < t1) {
          g4[u] = gk[tt];
          if (g4[u] != 0.0f && c < d / EPC) x4[u] = *reinterpret_cast<const u32x4*>(h + tt * d + c * EPC);
        }
      }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (g4[u] == 0.0f) continue;
        db += (double)g4[u];
        float x[EPC];
        unpack8<T>(x4[u], x);
#pragma unroll
        for (int e = 0; e < EPC; ++e) acc[e] = fmaf(g4[u], x[e], acc[e]);
      }
    }
    if (c < d / EPC) {
#pragma unroll
      for (int e = 0; e < EPC; ++e) part[(int64_t)blockIdx.x * d + c * EPC + e] = acc[e];
    }
    if (cb == 0 && threadIdx.x == 0) part_db[blockIdx.x] = db;
  }
}

// final sums over the workgroup partials in a fixed order (fp64): a block owns 32 columns; thread
// (column, part) adds the partials of its eighth of the workgroups in workgroup order, then the
// eight part sums of a column are added in part order.
__global__ void __launch_bounds__(256)
k_value_head_dw_final(int nblk, int d, const float* part, const double* part_db, float* dw, float* dbias) {
  __shared__ double sh[8][32];
  const int col = threadIdx.x & 31, pt = threadIdx.x >> 5;
  const int j = blockIdx.x * 32 + col;
  const int b0 = (int)((int64_t)nblk * pt / 8), b1 = (int)((int64_t)nblk * (pt + 1) / 8);
  double s = 0.0;
  if (j < d) {
#pragma unroll 8
    for (int b = b0; b < b1; ++b) s += (double)part[(int64_t)b * d + j];
  }
  sh[pt][col] = s;
  __syncthreads();
  if (pt == 0 && j < d) {
    double t = 0.0;
#pragma unroll
    for (int q = 0; q < 8; ++q) t += sh[q][col];
    dw[j] = (float)t;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    double t = 0.0;
    for (int b = 0; b < nblk; ++b) t += part_db[b];
    dbias[0] = (float)t;
  }
}

}  // namespace

size_t value_head_workspace(int64_t N, int d) {
  const int64_t nblk = (N + kHeadRows - 1) / kHeadRows;
  return (size_t)(((nblk * d * 4 + 255) / 256) * 256 + ((nblk * 8 + 255) / 256) * 256 + ((N * 4 + 255) / 256) * 256);
}

hipError_t launch_value_head_fwd(int dtype, int64_t N, int d, int R, const void* h, const void* w, float b,
                                 const uint8_t* mask, const int32_t* cu, const int32_t* gid, float* values,
                                 hipStream_t s) {
  if (N == 0) return hipSuccess;
  prof_mark(KK_VALUE_HEAD, true, s);
  const unsigned grid = (unsigned)((N + 3) / 4);
  if (dtype == RLK_DTYPE_BF16)
    k_value_head_fwd<bf16_t><<<grid, 256, 0, s>>>(N, d, (const bf16_t*)h, (const bf16_t*)w, b, mask, cu, gid, R,
                                                  values);
  else
    k_value_head_fwd<float><<<grid, 256, 0, s>>>(N, d, (const float*)h, (const float*)w, b, mask, cu, gid, R,
                                                 values);
  prof_mark(KK_VALUE_HEAD, false, s);
  return hipGetLastError();
}

hipError_t launch_value_head_bwd(int dtype, int64_t N, int d, int R, const void* h, const void* w,
                                 const uint8_t* mask, const int32_t* cu, const int32_t* gid, const float* dv,
                                 void* dh, int accumulate, float* dw, float* dbias, char* ws, hipStream_t s) {
  prof_mark(KK_VALUE_HEAD, true, s);
  const int64_t nblk64 = (N + kHeadRows - 1) / kHeadRows;
  const int nblk = (int)nblk64;
  float* part = reinterpret_cast<float*>(ws);
  const size_t part_bytes = ((nblk64 * d * 4 + 255) / 256) * 256;
  double* part_db = reinterpret_cast<double*>(ws + part_bytes);
  float* gk = reinterpret_cast<float*>(ws + part_bytes + ((nblk64 * 8 + 255) / 256) * 256);
  const bool bf = dtype == RLK_DTYPE_BF16;
  if (N > 0) {
    // dhidden rows (when dh is given) and every row's gradient gk for the sums below
    const unsigned grid = (unsigned)((N + 3) / 4);
    if (bf)
      k_value_head_dh<bf16_t><<<grid, 256, 0, s>>>(N, d, (const bf16_t*)w, dv, mask, cu, gid, R, (bf16_t*)dh,
                                                   accumulate, gk);
    else
      k_value_head_dh<float><<<grid, 256, 0, s>>>(N, d, (const float*)w, dv, mask, cu, gid, R, (float*)dh,
                                                  accumulate, gk);
  }
  if (nblk > 0) {
    if (bf)
      k_value_head_dw_partial<bf16_t><<<nblk, 256, 0, s>>>(N, d, (const bf16_t*)h, gk, part, part_db);
    else
      k_value_head_dw_partial<float><<<nblk, 256, 0, s>>>(N, d, (const float*)h, gk, part, part_db);
  }
  k_value_head_dw_final<<<(unsigned)((d + 31) / 32), 256, 0, s>>>(nblk, d, part, part_db, dw, dbias);
  prof_mark(KK_VALUE_HEAD, false, s);
  return hipGetLastError();
}

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
