// MFMA GEMMs of the LM-head projection and its two gradient contractions, with fused
// epilogues.  One core computes C[m][n] = sum_k A[m][k] * B[n][k] with both operands
// K-contiguous ("NT"); the three uses are
//   forward : A = W [V, d],          B = gathered hidden [tokens, d]   -> online log-softmax
//   dhidden : A = dz [tokens, Vp],   B = W^T [d, Vp]                   -> scatter to dh[idx]
//   dW      : A = dz^T [Vp, tokens], B = hidden^T [d, tokens]          -> fp32 dW (+)=
//
// Tile geometry (gfx950): 256 x 256 output tile per workgroup of 4 wavefronts (2 x 2), each
// wavefront owning 128 x 128 = 4 x 4 blocks of v_mfma_f32_32x32x16_bf16 (fp32 operands use
// v_mfma_f32_32x32x2_f32).  A stage holds 128 bytes of K per row (64 bf16 / 32 fp32) for both
// operands, staged through LDS with a 16-byte row pad (conflict-free 16-byte fragment
// reads) and double-buffered: 2 x 2 x 36 KiB = 144 KiB of the 160 KiB LDS.  Each lane's
// MFMA fragment carries 8 consecutive K elements of one row (16 bytes); A and B use the
// same K assignment, so the lane split of K inside the MFMA is irrelevant to the sum.
//
// Output layout of a 32x32 MFMA block: lane l holds column (l % 32); accumulator register r
// holds row 8*(r/4) + 4*(l/32) + (r%4).  With vocabulary on M and tokens on N, every lane's
// accumulators belong to a single token, so the vocabulary reduction of the online
// log-softmax is in-register, then one cross-half exchange, then one LDS exchange between
// the two wavefronts of a column.
//
// Workgroup-to-tile mapping is XCD-aware: consecutive workgroup ids are dispatched round-robin
// over the 8 XCDs, so ids are re-packed to give each XCD a contiguous range of tiles, which
// is then rastered in groups of 8 M-tiles so that concurrently resident tiles share operand
// panels in that XCD's L2.
#include "rlk_internal.h"

namespace rlk {

namespace {

constexpr int NT = 256;
constexpr int KB = 128;                 // bytes of K per stage per row
constexpr int LROW = KB + 16;           // LDS row stride (bytes)
constexpr int TILE_B = kTile * LROW;    // 36864
constexpr int STAGE_B = 2 * TILE_B;     // A + B
constexpr int LDS_B = 2 * STAGE_B;      // 147456
constexpr int QROW = kTile * 2 + 16;    // LDS row stride of the bf16 probability tile (bytes)
constexpr int RED_OFF = kTile * QROW;   // 135168: reduction scratch after the staged tile
constexpr int GROUP_M = 8;
constexpr float kLog2e = 1.4426950408889634f;

enum { EPI_FWD = 0, EPI_DH = 1, EPI_DW = 2 };

template <typename T>
struct Op;

template <>
struct Op<bf16_t> {
  static __device__ __forceinline__ void mma(f32x16& c, u32x4 a, u32x4 b) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c,
                                                0, 0, 0);
  }
};

template <>
struct Op<float> {
  static __device__ __forceinline__ void mma(f32x16& c, u32x4 a, u32x4 b) {
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.x), __uint_as_float(b.x), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.y), __uint_as_float(b.y), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.z), __uint_as_float(b.z), c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_32x32x2f32(__uint_as_float(a.w), __uint_as_float(b.w), c, 0, 0, 0);
  }
};

__device__ __forceinline__ uint16_t bf16_bits(float x) {
  return __builtin_bit_cast(uint16_t, (__bf16)x);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  bf16x2 v;
  v.x = (__bf16)lo;
  v.y = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

template <typename T>
__device__ __forceinline__ void store_elem(T* p, float x);
template <>
__device__ __forceinline__ void store_elem<float>(float* p, float x) { *p = x; }
template <>
__device__ __forceinline__ void store_elem<bf16_t>(bf16_t* p, float x) { p->bits = bf16_bits(x); }

// XCD-aware, L2-grouped tile mapping.  Returns false for workgroups beyond the tile grid.
__device__ __forceinline__ bool map_tile(int tm, int tn, int& tile_m, int& tile_n) {
  const int total = tm * tn;
  const int pid = blockIdx.x;
  if (pid >= total) return false;
  const int xcd = pid & 7, local = pid >> 3;
  const int base = total >> 3, rem = total & 7;
  const int start = xcd < rem ? xcd * (base + 1) : rem * (base + 1) + (xcd - rem) * base;
  const int npid = start + local;
  const int group_sz = GROUP_M * tn;
  const int g = npid / group_sz;
  const int first_m = g * GROUP_M;
  const int gm = min(tm - first_m, GROUP_M);
  const int in = npid - g * group_sz;
  tile_m = first_m + in % gm;
  tile_n = in / gm;
  return true;
}

template <typename T, int EPI, bool STORE_Q>
__global__ void __launch_bounds__(NT, 1) k_gemm(GemmArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[LDS_B];

  int M = a.M, N = a.N, K = a.K;
  int64_t rc = (int64_t)a.hdr->n_eff - a.c0;
  rc = rc < 0 ? 0 : (rc > a.Mc ? a.Mc : rc);
  if (EPI == EPI_FWD) N = (int)rc;
  if (EPI == EPI_DH) M = (int)rc;
  if (EPI == EPI_DW) {
    if (rc == 0 && a.c0 > 0) return;  // nothing to add from an empty chunk
    K = (int)((rc + kKAlign - 1) / kKAlign * kKAlign);
  }
  if (M <= 0 || N <= 0) return;
  const int tm = (M + kTile - 1) / kTile, tn = (N + kTile - 1) / kTile;
  int tile_m, tile_n;
  if (!map_tile(tm, tn, tile_m, tile_n)) return;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wid = tid >> 6, wm = wid >> 1, wn = wid & 1;
  const int lrow = lane & 31, lh = lane >> 5;

  // ---- operand row pointers for the global->LDS copy: rows (tid>>3) + 32 i, 16-byte column tid&7
  const int64_t lda_b = a.lda * (int64_t)sizeof(T), ldb_b = a.ldb * (int64_t)sizeof(T);
  const char* pa[8];
  const char* pb[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    int ra = min(tile_m * kTile + (tid >> 3) + 32 * i, M - 1);
    int rb = min(tile_n * kTile + (tid >> 3) + 32 * i, N - 1);
    pa[i] = reinterpret_cast<const char*>(a.A) + (int64_t)ra * lda_b + (tid & 7) * 16;
    pb[i] = reinterpret_cast<const char*>(a.B) + (int64_t)rb * ldb_b + (tid & 7) * 16;
  }
  const int64_t Kb = (int64_t)K * sizeof(T);
  const int nk = (int)((Kb + KB - 1) / KB);

  u32x4 ra[8], rb[8];
  auto gload = [&](int kt) {
    const int64_t kb = (int64_t)kt * KB;
    const bool ok = kb + (tid & 7) * 16 < Kb;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      if (ok) {
        ra[i] = *reinterpret_cast<const u32x4*>(pa[i] + kb);
        rb[i] = *reinterpret_cast<const u32x4*>(pb[i] + kb);
      } else {
        ra[i] = u32x4{0, 0, 0, 0};
        rb[i] = u32x4{0, 0, 0, 0};
      }
    }
  };
  auto sstore = [&](int buf) {
    char* sA = smem + buf * STAGE_B;
    char* sB = sA + TILE_B;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int off = ((tid >> 3) + 32 * i) * LROW + (tid & 7) * 16;
      *reinterpret_cast<u32x4*>(sA + off) = ra[i];
      *reinterpret_cast<u32x4*>(sB + off) = rb[i];
    }
  };

  f32x16 acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) gload(kt + 1);
    const char* sA = smem + (kt & 1) * STAGE_B;
    const char* sB = sA + TILE_B;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      u32x4 af[4], bfr[4];
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
        af[mb] = *reinterpret_cast<const u32x4*>(sA + (wm * 128 + mb * 32 + lrow) * LROW + kk * 32 + lh * 16);
#pragma unroll
      for (int nb = 0; nb < 4; ++nb)
        bfr[nb] = *reinterpret_cast<const u32x4*>(sB + (wn * 128 + nb * 32 + lrow) * LROW + kk * 32 + lh * 16);
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int nb = 0; nb < 4; ++nb) Op<T>::mma(acc[mb][nb], af[mb], bfr[nb]);
    }
    if (kt + 1 < nk) sstore((kt + 1) & 1);
    __syncthreads();
  }

  // ------------------------------------------------------------------ epilogues
  if constexpr (EPI == EPI_FWD) {
    // rows = vocabulary v = v0 + rl, columns = chunk-local token n.
    const int v0 = tile_m * kTile;
    const int V = a.V;
    const bool full_v = v0 + kTile <= V;
    float* red_m = reinterpret_cast<float*>(smem + RED_OFF);  // [2][256]
    float* red_s = red_m + 2 * kTile;                          // [2][256]
    float* red_u = red_s + 2 * kTile;                          // [2][256]

    // phase 1: per-token max over this tile's 256 vocabulary rows; gather the target logit.
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      const int cl = wn * 128 + nb * 32 + lrow;
      const int n = tile_n * kTile + cl;
      float mx = -INFINITY;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rl = wm * 128 + mb * 32 + (r >> 2) * 8 + lh * 4 + (r & 3);
          const float z = (full_v || v0 + rl < V) ? acc[mb][nb][r] : -INFINITY;
          mx = fmaxf(mx, z);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      if (lh == 0) red_m[wm * kTile + cl] = mx;
      if (n < N) {
        const int y = a.ytgt[a.c0 + n];
        const int yl = y - v0 - wm * 128;
        if (y >= 0 && y < V && yl >= 0 && yl < 128 && ((yl >> 2) & 1) == lh) {
          const int tmb = yl >> 5, tr = ((yl & 31) >> 3) * 4 + (yl & 3);
          float z = 0.0f;
#pragma unroll
          for (int mb = 0; mb < 4; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) z = (mb == tmb && r == tr) ? acc[mb][nb][r] : z;
          a.zy[a.c0 + n] = z;
        }
      }
    }
    __syncthreads();

    // phase 2: e = exp(z - m), s = sum e, u = sum e (z - m); e optionally staged for storage.
    char* sQ = smem;
#pragma unroll
    for (int nb = 0; nb < 4; ++nb) {
      const int cl = wn * 128 + nb * 32 + lrow;
      const float mt = fmaxf(red_m[cl], red_m[kTile + cl]);
      const float mt2 = mt * kLog2e;
      float s = 0.0f, u = 0.0f;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float ev[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int r = g * 4 + i;
            const int rl = wm * 128 + mb * 32 + g * 8 + lh * 4 + i;
            const float z = acc[mb][nb][r];
            const bool valid = full_v || v0 + rl < V;
            const float e = valid ? __builtin_amdgcn_exp2f(fmaf(z, kLog2e, -mt2)) : 0.0f;
            s += e;
            u = fmaf(e, z - mt, u);
            ev[i] = e;
          }
          if constexpr (STORE_Q) {
            if constexpr (sizeof(T) == 2) {
              const int rl0 = wm * 128 + mb * 32 + g * 8 + lh * 4;
              u32x2 pk;
              pk.x = pack_bf16x2(ev[0], ev[1]);
              pk.y = pack_bf16x2(ev[2], ev[3]);
              *reinterpret_cast<u32x2*>(sQ + cl * QROW + rl0 * 2) = pk;
            } else {
              const int n = tile_n * kTile + cl;
              if (n < N) {
                const int rl0 = wm * 128 + mb * 32 + g * 8 + lh * 4;
                float* qp = reinterpret_cast<float*>(a.q) + (int64_t)n * a.ldq + v0 + rl0;
#pragma unroll
                for (int i = 0; i < 4; ++i) qp[i] = ev[i];
              }
            }
          }
        }
      s += __shfl_xor(s, 32, 64);
      u += __shfl_xor(u, 32, 64);
      if (lh == 0) {
        red_s[wm * kTile + cl] = s;
        red_u[wm * kTile + cl] = u;
      }
    }
    __syncthreads();
    if (wm == 0 && lh == 0) {
#pragma unroll
      for (int nb = 0; nb < 4; ++nb) {
        const int cl = wn * 128 + nb * 32 + lrow;
        const int n = tile_n * kTile + cl;
        if (n < N) {
          const int64_t o = (int64_t)tile_m * a.Mc + n;
          a.pm[o] = fmaxf(red_m[cl], red_m[kTile + cl]);
          a.ps[o] = red_s[cl] + red_s[kTile + cl];
          a.pu[o] = red_u[cl] + red_u[kTile + cl];
        }
      }
    }
    if constexpr (STORE_Q && sizeof(T) == 2) {
      // phase 3: coalesced copy of the staged bf16 tile to q[n][v0 .. v0 + 255].
      const int chunk = tid & 31;
#pragma unroll 4
      for (int it = 0; it < 32; ++it) {
        const int cl = (tid >> 5) + 8 * it;
        const int n = tile_n * kTile + cl;
        if (n < N) {
          const u32x4 v = *reinterpret_cast<const u32x4*>(sQ + cl * QROW + chunk * 16);
          char* dst = reinterpret_cast<char*>(a.q) + ((int64_t)n * a.ldq + v0) * 2 + chunk * 16;
          *reinterpret_cast<u32x4*>(dst) = v;
        }
      }
    }
  } else if constexpr (EPI == EPI_DH) {
    // rows = chunk-local tokens, columns = hidden features; scatter to dh[idx[c0 + row]].
    T* out = reinterpret_cast<T*>(a.out);
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = tile_m * kTile + wm * 128 + mb * 32 + (r >> 2) * 8 + lh * 4 + (r & 3);
        if (rl < M) {
          const int64_t row = a.idx[a.c0 + rl];
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) {
            const int cl = tile_n * kTile + wn * 128 + nb * 32 + lrow;
            if (cl < N) store_elem<T>(out + row * a.ldo + cl, acc[mb][nb][r]);
          }
        }
      }
  } else {
    // rows = vocabulary, columns = hidden features; fp32 dW, overwritten by the first
    // chunk unless the caller accumulates.
    const bool add = a.accumulate || a.c0 > 0;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = tile_m * kTile + wm * 128 + mb * 32 + (r >> 2) * 8 + lh * 4 + (r & 3);
        if (rl < M) {
#pragma unroll
          for (int nb = 0; nb < 4; ++nb) {
            const int cl = tile_n * kTile + wn * 128 + nb * 32 + lrow;
            if (cl < N) {
              float* p = a.dw + (int64_t)rl * a.ldo + cl;
              *p = add ? *p + acc[mb][nb][r] : acc[mb][nb][r];
            }
          }
        }
      }
  }
}

inline unsigned tiles(int64_t n) { return (unsigned)((n + kTile - 1) / kTile); }

template <typename T>
hipError_t fwd_impl(const GemmArgs& a, bool store_q, hipStream_t s) {
  dim3 grid(tiles(a.M) * tiles(a.Mc));
  if (store_q)
    k_gemm<T, EPI_FWD, true><<<grid, NT, 0, s>>>(a);
  else
    k_gemm<T, EPI_FWD, false><<<grid, NT, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_fwd_gemm(int dtype, const GemmArgs& a, bool store_q, hipStream_t s) {
  prof_mark(KK_FWD_GEMM, true, s);
  hipError_t e = dtype == RLK_DTYPE_BF16 ? fwd_impl<bf16_t>(a, store_q, s) : fwd_impl<float>(a, store_q, s);
  prof_mark(KK_FWD_GEMM, false, s);
  return e;
}

hipError_t launch_dh_gemm(int dtype, const GemmArgs& a, hipStream_t s) {
  dim3 grid(tiles(a.Mc) * tiles(a.N));
  prof_mark(KK_DH_GEMM, true, s);
  if (dtype == RLK_DTYPE_BF16)
    k_gemm<bf16_t, EPI_DH, false><<<grid, NT, 0, s>>>(a);
  else
    k_gemm<float, EPI_DH, false><<<grid, NT, 0, s>>>(a);
  prof_mark(KK_DH_GEMM, false, s);
  return hipGetLastError();
}

hipError_t launch_dw_gemm(int dtype, const GemmArgs& a, hipStream_t s) {
  dim3 grid(tiles(a.M) * tiles(a.N));
  prof_mark(KK_DW_GEMM, true, s);
  if (dtype == RLK_DTYPE_BF16)
    k_gemm<bf16_t, EPI_DW, false><<<grid, NT, 0, s>>>(a);
  else
    k_gemm<float, EPI_DW, false><<<grid, NT, 0, s>>>(a);
  prof_mark(KK_DW_GEMM, false, s);
  return hipGetLastError();
}

}  // namespace rlk
