// Per-token kernels of the hot path: operand gathers/transposes, the merge of the online
// log-softmax partials, the loss terms and their per-token backward scalars, the logits
// gradient dz, the deterministic loss reduction and the zero fill of untrained rows.
//
// Notation (ClawGym II, Sec. 2.3): z = W h, lse = logsumexp(z), logp = z_y - lse,
// H = -sum_j p_j log p_j, rho = exp(logp - old_logp), A = group advantage of the token's
// rollout, s = min(rho A, clip(rho, 1-eps_lo, 1+eps_hi) A), loss L = sum_t w_t (s_t + c H_t)
// with w_t = -1/(Q G_q n_r) for the per-rollout/per-group mean (masked GRPO objective,
// Sec. 2.3.2 with the tree rule of Sec. 3.2.3) or -1/sum M for the token mean (Sec. 2.3.1).
// Backward: dL/dlogp_t = g_t = w_t A rho_t [not clipped], dL/dH_t = e_t = w_t c, and
//   dz_tj = g_t ([j = y_t] - p_tj) - e_t p_tj (z_tj - lse_t + H_t).
// Optional terms: truncated importance sampling (Sec. 3.2.4) multiplies w_t by
// min(exp(old_t - rollout_t), c_bar); the KL term of the GRPO objective (Sec. 2.3.2) adds
// -beta (e^r - r - 1), r = ref_t - logp_t, to the token's objective, so g_t gains w_t beta (e^r - 1).
#include "rlk_internal.h"

#include <algorithm>

namespace rlk {

namespace {

constexpr float kLog2e = 1.4426950408889634f;
constexpr int64_t kDzBlocks = 8192;  // grid of the flagged-chunk dz launch (32 blocks per CU)

__device__ __forceinline__ float bf16_to_f(uint16_t b) { return __uint_as_float(((uint32_t)b) << 16); }
__device__ __forceinline__ uint16_t f_to_bf16(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }

template <typename X>
__device__ inline X wave_sum(X v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// 16-byte vectors of 8 bf16 (stored as uint16_t bit patterns) or 4 fp32 elements.
template <typename T>
__device__ __forceinline__ float vget(const u32x4& v, int k) {
  if constexpr (sizeof(T) == 2) {
    const uint32_t w = v[k >> 1];
    return bf16_to_f((uint16_t)((k & 1) ? (w >> 16) : (w & 0xffffu)));
  } else {
    return __uint_as_float(v[k]);
  }
}

template <typename T>
__device__ __forceinline__ T to_storage(float x) {
  if constexpr (sizeof(T) == 2) return f_to_bf16(x);
  else return x;
}

template <typename T>
__device__ __forceinline__ u32x4 vpack(const T* e) {
  u32x4 v;
  if constexpr (sizeof(T) == 2) {
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = (uint32_t)e[2 * j] | ((uint32_t)e[2 * j + 1] << 16);
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = __float_as_uint(e[j]);
  }
  return v;
}

// ---- W^T [d][ldw] (columns v < Vp; zero beyond V) for the dhidden GEMM, 64 x 64 tiles through LDS
// with 16-byte global loads and stores: a thread reads 16 bytes along a row of W and writes 16
// bytes (EPC consecutive vocabulary entries) along a row of W^T.
template <typename T>
__global__ void __launch_bounds__(256) k_transpose_w(const T* W, T* WT, int V, int64_t Vp, int d, int64_t ldw) {
  constexpr int EPC = 16 / sizeof(T);
  constexpr int CPR = 64 / EPC;  // 16-byte chunks per 64-element tile row
  __shared__ T tile[64][64 + 2];
  const int64_t v0 = (int64_t)blockIdx.x * 64;
  const int j0 = blockIdx.y * 64;
  for (int c = threadIdx.x; c < 64 * CPR; c += 256) {
    const int r = c / CPR, ch = c % CPR;  // vocabulary row r, feature chunk ch
    const int64_t v = v0 + r;
    const int j = j0 + ch * EPC;
    T vals[EPC];
    if (v < V && j + EPC <= d) {
      const u32x4 x = *reinterpret_cast<const u32x4*>(W + v * d + j);
#pragma unroll
      for (int e = 0; e < EPC; ++e) vals[e] = reinterpret_cast<const T*>(&x)[e];
    } else {
#pragma unroll
      for (int e = 0; e < EPC; ++e) vals[e] = (v < V && j + e < d) ? W[v * d + j + e] : T(0);
    }
#pragma unroll
    for (int e = 0; e < EPC; ++e) tile[r][ch * EPC + e] = vals[e];
  }
  __syncthreads();
  for (int c = threadIdx.x; c < 64 * CPR; c += 256) {
    const int jr = c / CPR, ch = c % CPR;  // feature row jr of W^T, vocabulary chunk ch
    const int j = j0 + jr;
    const int64_t v = v0 + ch * EPC;
    if (j >= d || v >= Vp) continue;
    T vals[EPC];
#pragma unroll
    for (int e = 0; e < EPC; ++e) vals[e] = tile[ch * EPC + e][jr];
    *reinterpret_cast<u32x4*>(WT + (int64_t)j * ldw + v) = vpack<T>(vals);
  }
}

// ---- Hc[t][:] = hidden[idx[c0 + t]][:] and HT[j][t] (row stride ldt; zero columns t >= rows, up to
// the K pad).
template <typename T>
__global__ void __launch_bounds__(256)
k_gather(const T* hidden, int d, const int32_t* idx, const WsHeader* hdr, int64_t c0, int64_t Mc, T* hc, T* ht,
         int64_t ldt, int want_ht) {
  constexpr int EPC = 16 / sizeof(T);     // elements per 16-byte chunk
  constexpr int CPR = 64 / EPC;           // chunks per 64-feature row slice
  __shared__ __attribute__((aligned(16))) T tile[64][64 + EPC];
  int64_t rc = (int64_t)hdr->n_eff - c0;
  rc = rc < 0 ? 0 : (rc > Mc ? Mc : rc);
  const int64_t rpad = (rc + kKAlign - 1) / kKAlign * kKAlign;
  const int64_t t0 = (int64_t)blockIdx.x * 64;
  const int j0 = blockIdx.y * 64;
  if (t0 >= rpad) return;
  for (int c = threadIdx.x; c < 64 * CPR; c += 256) {
    const int tl = c / CPR, ch = c % CPR;
    const int64_t t = t0 + tl;
    const int j = j0 + ch * EPC;
    u32x4 v = u32x4{0, 0, 0, 0};
    if (t < rc && j < d) {
      const int64_t row = idx[c0 + t];
      v = *reinterpret_cast<const u32x4*>(hidden + row * d + j);
      *reinterpret_cast<u32x4*>(hc + t * d + j) = v;
    }
    *reinterpret_cast<u32x4*>(&tile[tl][ch * EPC]) = v;
  }
  if (!want_ht) return;
  __syncthreads();
  for (int c = threadIdx.x; c < 64 * CPR; c += 256) {
    const int jl = c / CPR, ch = c % CPR;   // feature row of HT, chunk of 8/4 tokens
    const int j = j0 + jl;
    if (j >= d) continue;
    T vals[EPC];
#pragma unroll
    for (int i = 0; i < EPC; ++i) vals[i] = tile[ch * EPC + i][jl];
    *reinterpret_cast<u32x4*>(ht + (int64_t)j * ldt + t0 + ch * EPC) = vpack<T>(vals);
  }
}

// ---- reference logits of the token-reference layout (bf16): zr[t] = (hc[t] . W[y_t]) / tau, one
// wavefront per chunk row, fp32 sums of 16-byte loads.  Block 0 also clears the chunk's flag.
__global__ void __launch_bounds__(256) k_target_logit(const uint16_t* hc, int d, const uint16_t* W,
                                                      const int32_t* ytgt, const WsHeader* hdr, int64_t c0,
                                                      int64_t Mc, int V, float inv_tau, float* zr, int32_t* fb) {
  if (blockIdx.x == 0 && threadIdx.x == 0) *fb = 0;
  int64_t rc = (int64_t)hdr->n_eff - c0;
  rc = rc < 0 ? 0 : (rc > Mc ? Mc : rc);
  const int lane = threadIdx.x & 63;
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= rc) return;
  const int y = ytgt[c0 + t];
  float acc = 0.0f;
  if (y >= 0 && y < V) {
    const uint16_t* h = hc + t * d;
    const uint16_t* w = W + (int64_t)y * d;
    for (int j = lane * 8; j < d; j += 512) {
      const u32x4 x = *reinterpret_cast<const u32x4*>(h + j);
      const u32x4 v = *reinterpret_cast<const u32x4*>(w + j);
#pragma unroll
      for (int k = 0; k < 8; ++k) acc = fmaf(vget<uint16_t>(x, k), vget<uint16_t>(v, k), acc);
    }
  }
  acc = wave_sum(acc);
  if (lane == 0) zr[t] = acc * inv_tau;
}

// ---- HT[j][t] = hc[t][j] * s_t for the dW GEMM of the token-reference layout (s_t = 1 when the
// chunk is flagged); zero columns t in [rows, K pad).  64 x 64 tiles through LDS as in k_gather.
__global__ void __launch_bounds__(256) k_hidden_t(const uint16_t* hc, int d, const float* st, const int32_t* fb,
                                                  const WsHeader* hdr, int64_t c0, int64_t Mc, uint16_t* ht,
                                                  int64_t ldt) {
  __shared__ __attribute__((aligned(16))) uint16_t tile[64][64 + 8];
  int64_t rc = (int64_t)hdr->n_grad - c0;  // rows with a surrogate gradient
  rc = rc < 0 ? 0 : (rc > Mc ? Mc : rc);
  const int64_t rpad = (rc + kKAlign - 1) / kKAlign * kKAlign;
  const int64_t t0 = (int64_t)blockIdx.x * 64;
  const int j0 = blockIdx.y * 64;
  if (t0 >= rpad) return;
  const bool scaled = *fb == 0;
  for (int c = threadIdx.x; c < 64 * 8; c += 256) {
    const int tl = c / 8, ch = c % 8;
    const int64_t t = t0 + tl;
    const int j = j0 + ch * 8;
    u32x4 v = u32x4{0, 0, 0, 0};
    if (t < rc && j < d) {
      v = *reinterpret_cast<const u32x4*>(hc + t * d + j);
      if (scaled) {
        const float sc = st[t];
        uint16_t e[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) e[k] = f_to_bf16(vget<uint16_t>(v, k) * sc);
        v = vpack<uint16_t>(e);
      }
    }
    *reinterpret_cast<u32x4*>(&tile[tl][ch * 8]) = v;
  }
  __syncthreads();
  for (int c = threadIdx.x; c < 64 * 8; c += 256) {
    const int jl = c / 8, ch = c % 8;
    const int j = j0 + jl;
    if (j >= d) continue;
    uint16_t vals[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) vals[i] = tile[ch * 8 + i][jl];
    *reinterpret_cast<u32x4*>(ht + (int64_t)j * ldt + t0 + ch * 8) = vpack<uint16_t>(vals);
  }
}

// ---- merge of the per-vocabulary-tile partials (m, s, u) into lse, logp, H; loss scalars.
__global__ void __launch_bounds__(256) k_combine(TokenParams p) {
  // 64 tokens per block; wavefront w merges the vocabulary tiles k = w, w + 4, ... of its lane's
  // token (loads coalesced over the 64 tokens) in one pass with a running maximum M_w:
  //   S_w = sum_k e^{m_k - M_w} s_k,  T_w = sum_k e^{m_k - M_w} (u_k + (m_k - M_w) s_k),
  // rescaled by e^{M_w - M'} (and T_w shifted by (M_w - M') S_w) whenever the maximum grows to M';
  // the four wavefront results meet in LDS the same way.  Then lse = M + ln S and
  // sum_j p_j (z_j - lse) = T / S - ln S.
  __shared__ float s_m[4][64];
  __shared__ double s_S[4][64], s_T[4][64];
  int64_t rc = (int64_t)p.hdr->n_eff - p.c0;
  rc = rc < 0 ? 0 : (rc > p.Mc ? p.Mc : rc);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const int64_t tl = (int64_t)blockIdx.x * 64 + lane;
  if ((int64_t)blockIdx.x * 64 >= rc) return;
  const bool act = tl < rc;
  float Mw = -INFINITY;
  double S = 0.0, T = 0.0;
  if (act)
    for (int k = wv; k < p.nvt; k += 4) {
      const int64_t o = (int64_t)k * p.Mc + tl;
      const float mk = p.pm[o];
      const double sk = (double)p.ps[o];
      const double uk = (double)p.pu[o];
      if (mk > Mw) {
        if (Mw > -INFINITY) {
          const double f = (double)__builtin_amdgcn_exp2f((Mw - mk) * kLog2e);
          T = f * (T + (double)(Mw - mk) * S);
          S *= f;
        }
        Mw = mk;
      }
      const double w = (double)__builtin_amdgcn_exp2f((mk - Mw) * kLog2e);
      S += w * sk;
      T += w * (uk + (double)(mk - Mw) * sk);
    }
  s_m[wv][lane] = Mw;
  s_S[wv][lane] = S;
  s_T[wv][lane] = T;
  __syncthreads();
  if (wv != 0 || !act) return;
  const float M = fmaxf(fmaxf(s_m[0][lane], s_m[1][lane]), fmaxf(s_m[2][lane], s_m[3][lane]));
  S = 0.0;
  T = 0.0;
#pragma unroll
  for (int w4 = 0; w4 < 4; ++w4) {
    const float mw = s_m[w4][lane];
    if (mw == -INFINITY) continue;  // a wavefront without vocabulary tiles (fewer than 4 tiles)
    const double f = (double)__builtin_amdgcn_exp2f((mw - M) * kLog2e);
    S += f * s_S[w4][lane];
    T += f * (s_T[w4][lane] + (double)(mw - M) * s_S[w4][lane]);
  }
  const int64_t i = p.c0 + tl;
  const double lnS = log(S);
  const double lse = (double)M + lnS;
  const double E = T / S - lnS;
  const float lsef = (float)lse;
  const float H = (float)(-E);
  const float logp = (float)((double)p.zy[i] - lse);
  p.lse[i] = lsef;
  p.logp[i] = logp;
  p.ent[i] = H;
  const int64_t row = p.idx[i];
  if (p.logp_out) p.logp_out[row] = logp;
  if (p.ent_out) p.ent_out[row] = H;
  if (p.lse_out) p.lse_out[row] = lsef;
  if (p.with_grad) {
    const int r = p.tokr[i];
    const float A = p.token_adv ? p.token_adv[row] : p.adv[r];
    const float old = p.old_logp[row];
    const float rho = expf(logp - old);
    double w;
    if (p.agg == RLK_AGG_SEQ_MEAN_TOKEN_MEAN) {
      const double Qn = p.norm_override > 0 ? p.norm_override : (double)p.hdr->n_groups;
      w = -1.0 / (Qn * (double)p.gsize[p.gidx[r]] * (double)p.rnpol[r]);
    } else {
      const double Mn = p.norm_override > 0 ? p.norm_override : (double)p.hdr->n_eff;
      w = -1.0 / Mn;
    }
    // truncated importance weight (Sec. 3.2.4): a constant factor on the token's whole loss
    if (p.rollout_logp) w *= (double)fminf(expf(old - p.rollout_logp[row]), p.tis_cap);
    const bool clipped = (A > 0.0f && rho > 1.0f + p.eps_high) || (A < 0.0f && rho < 1.0f - p.eps_low);
    double dlogp = clipped ? 0.0 : (double)A * (double)rho;
    // KL term: d/dlogp of -beta (e^r - r - 1), r = ref - logp, is beta (e^r - 1)
    if (p.ref_logp) dlogp += (double)p.kl_coef * (double)expm1f(p.ref_logp[row] - logp);
    // g, e are taken per raw logit W h: the temperature's 1 / tau enters here, once
    const float g = (float)(w * dlogp * (double)p.inv_tau);
    p.gt[i] = g;
    p.et[i] = (float)(w * (double)p.ent_coef * (double)p.inv_tau);
    if (p.zr) {
      // Token-reference layout: q_tj = exp(z_tj - r), so dz_tj = -g p_tj = s q_tj with
      // s = -g exp(r - lse), except at the target, where dz = g (1 - p_y) = -g expm1(logp): its
      // entry of q and q^T becomes expm1(logp) exp(lse - r), and dz = diag(s) q holds exactly.
      const float r = p.zr[tl];
      const float sc = -g * expf(r - lsef);
      const float qy = expm1f(logp) * expf(lsef - r);
      p.st[tl] = sc;
      if (!(fabsf(qy) <= kRefQMax) || (sc != 0.0f && !(fabsf(sc) >= kRefSMin))) *p.fb = 1;
      const int y = p.ytgt[i];
      if (y >= 0 && y < p.V) {
        const uint16_t qb = f_to_bf16(qy);
        reinterpret_cast<uint16_t*>(p.q)[tl * p.ldq + y] = qb;
        reinterpret_cast<uint16_t*>(p.qt)[(int64_t)y * p.ldqt + tl] = qb;
      }
    }
  }
}

// ---- dz for a chunk: q holds exp(z - c) per (token, vocabulary) against the reference c = pm of
// its (token, vocabulary tile); rewritten in place with dz and also written transposed for the dW
// GEMM.  Block tile: 64 tokens x 256 vocabulary entries (one forward vocabulary tile, so one c
// per token).  Each thread owns an EPC x EPC
// square (EPC tokens x EPC consecutive vocabulary entries, EPC = elements per 16 bytes): it reads
// EPC 16-byte rows, writes them back as dz and transposes the square in registers into EPC
// 16-byte rows of dz^T, so neither layout needs an LDS pass.  The per-token scalars are
// computed once per block tile into LDS.
// One block tile: tokens t0 .. t0 + 63 of the chunk, vocabulary tile vt.
struct DzShared {
  float sc[64], g[64], e[64], base[64], dzy[64];
  int y[64], ok[64];   // ok: token inside the chunk (else dz = 0)
};

template <typename T, bool ENT>
__device__ __forceinline__ void dz_tile(const DzParams& p, int vt, int64_t t0, int64_t rc, DzShared& sh) {
  constexpr int EPC = 16 / sizeof(T);
  constexpr int TG = 64 / EPC;                  // token groups per block (lanes along tokens)
  constexpr int VC = 64 / TG;                   // vocabulary chunks per wavefront pass
  constexpr int VSPAN = VC * EPC;               // vocabulary entries per wavefront pass
  constexpr int PASSES = kVocabTile / (4 * VSPAN);
  const int64_t v0 = (int64_t)vt * kVocabTile;
  if (threadIdx.x < 64) {
    const int tl = threadIdx.x;
    const int64_t t = t0 + tl;
    float sc = 0.0f, g = 0.0f, e = 0.0f, base = 0.0f, dzy = 0.0f;
    int y = -1;
    if (t < rc) {
      const int64_t i = p.c0 + t;
      const float lse = p.lse[i], logp = p.logp[i], H = p.ent[i];
      g = p.gt[i];
      e = p.et[i];
      const float mk = p.pm[(int64_t)vt * p.Mc + t];
      sc = __builtin_amdgcn_exp2f((mk - lse) * kLog2e);
      base = mk - lse + H;    // z - lse + H = log q + base
      const int yy = p.ytgt[i];
      if (yy >= v0 && yy < v0 + kVocabTile) y = (int)(yy - v0);
      // the target entry uses the exact fp32 log-prob: 1 - p_y = -expm1(logp)
      dzy = g * (-expm1f(logp));
      if (ENT) dzy -= e * expf(logp) * (logp + H);
    }
    sh.sc[tl] = sc;
    sh.g[tl] = g;
    sh.e[tl] = e;
    sh.base[tl] = base;
    sh.dzy[tl] = dzy;
    sh.y[tl] = y;
    sh.ok[tl] = t < rc;
  }
  __syncthreads();
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  const int vc = lane % VC, tg = lane / VC;
  T* q = reinterpret_cast<T*>(p.q);
  T* dzt = reinterpret_cast<T*>(p.dzt);
#pragma unroll
  for (int ps = 0; ps < PASSES; ++ps) {
    const int vl0 = (ps * 4 + wid) * VSPAN + vc * EPC;   // tile-local first vocabulary entry
    u32x4 raw[EPC];
#pragma unroll
    for (int j = 0; j < EPC; ++j)
      raw[j] = *reinterpret_cast<const u32x4*>(q + (t0 + tg * EPC + j) * p.ldq + v0 + vl0);
    float o[EPC][EPC];
#pragma unroll
    for (int j = 0; j < EPC; ++j) {
      const int tl = tg * EPC + j;
      const float sc = sh.sc[tl], g = sh.g[tl];
      const int y = sh.y[tl];
      const bool ok = sh.ok[tl] != 0;
#pragma unroll
      for (int k = 0; k < EPC; ++k) {
        const float qv = vget<T>(raw[j], k);
        float coef = g;
        if (ENT) coef += (qv > 0.0f) ? sh.e[tl] * (__logf(qv) + sh.base[tl]) : 0.0f;
        o[j][k] = !ok ? 0.0f : (vl0 + k == y) ? sh.dzy[tl] : -(qv * sc) * coef;
      }
    }
#pragma unroll
    for (int j = 0; j < EPC; ++j) {
      T row[EPC];
#pragma unroll
      for (int k = 0; k < EPC; ++k) row[k] = to_storage<T>(o[j][k]);
      *reinterpret_cast<u32x4*>(q + (t0 + tg * EPC + j) * p.ldq + v0 + vl0) = vpack<T>(row);
    }
#pragma unroll
    for (int k = 0; k < EPC; ++k) {
      T col[EPC];
#pragma unroll
      for (int j = 0; j < EPC; ++j) col[j] = to_storage<T>(o[j][k]);
      *reinterpret_cast<u32x4*>(dzt + (v0 + vl0 + k) * p.ldt + t0 + tg * EPC) = vpack<T>(col);
    }
  }
}

// One block per block tile (vocabulary tiles along x): a looping grid measured 22 % slower (the loop
// cost registers and a wave of occupancy).
template <typename T, bool ENT>
__global__ void __launch_bounds__(256, 5) k_dz(DzParams p) {
  if (p.ndz && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) atomicAdd(p.ndz, 1);
  int64_t rc = (int64_t)p.hdr->n_grad - p.c0;  // rows with a surrogate gradient
  rc = rc < 0 ? 0 : (rc > p.Mc ? p.Mc : rc);
  const int64_t rpad = (rc + kKAlign - 1) / kKAlign * kKAlign;
  const int64_t t0 = (int64_t)blockIdx.y * 64;
  if (t0 >= rpad) return;
  __shared__ DzShared sh;
  dz_tile<T, ENT>(p, blockIdx.x, t0, rc, sh);
}

// The same for a chunk of the token-reference layout (no entropy term), where dz = diag(s) q is
// applied by the GEMMs: nothing unless the chunk is flagged, so an unflagged chunk costs one small
// grid of empty blocks; the blocks of that grid loop over the block tiles.
template <typename T>
__global__ void __launch_bounds__(256) k_dz_flagged(DzParams p) {
  if (*p.fb == 0) return;
  if (p.ndz && blockIdx.x == 0 && threadIdx.x == 0) atomicAdd(p.ndz, 1);
  int64_t rc = (int64_t)p.hdr->n_grad - p.c0;  // rows with a surrogate gradient
  rc = rc < 0 ? 0 : (rc > p.Mc ? p.Mc : rc);
  const int64_t rpad = (rc + kKAlign - 1) / kKAlign * kKAlign;
  const int nvt = (int)(p.Vp / kVocabTile);
  const int64_t nbt = (int64_t)nvt * (rpad / 64);
  __shared__ DzShared sh;
  for (int64_t bt = blockIdx.x; bt < nbt; bt += gridDim.x) {
    dz_tile<T, false>(p, (int)(bt % nvt), bt / nvt * 64, rc, sh);
    __syncthreads();  // the next block tile rewrites the per-token scalars
  }
}

// ---- deterministic loss reduction: per-rollout fp64 sums, then one block over rollouts.
// Per-rollout sums: [0] w s, [1] w H, [2] w KL (the loss terms, w = importance weight or 1),
// [3] H, [4] rho, [5] clipped, [6] KL, [7] w (statistics).
__global__ void __launch_bounds__(256) k_loss_rollout(LossParams p) {
  __shared__ double sh[4][kRollSums];
  const int r = blockIdx.x;
  const int n = p.rnpol[r];
  const int s0 = p.rstart[r];
  const float Ar = p.adv[r];
  double acc[kRollSums];
#pragma unroll
  for (int f = 0; f < kRollSums; ++f) acc[f] = 0.0;
  if (p.gidx[r] >= 0) {
    for (int k = threadIdx.x; k < n; k += 256) {
      const int i = s0 + k;
      const int64_t row = p.idx[i];
      const float A = p.token_adv ? p.token_adv[row] : Ar;
      const float logp = p.logp[i];
      const float old = p.old_logp[row];
      const float rho = expf(logp - old);
      const float lo = 1.0f - p.eps_low, hi = 1.0f + p.eps_high;
      const float cr = fminf(fmaxf(rho, lo), hi);
      const float s = fminf(rho * A, cr * A);
      const bool clipped = (A > 0.0f && rho > hi) || (A < 0.0f && rho < lo);
      const double w = p.rollout_logp ? (double)fminf(expf(old - p.rollout_logp[row]), p.tis_cap) : 1.0;
      double kl = 0.0;
      if (p.ref_logp) {
        const float d = p.ref_logp[row] - logp;
        kl = (double)expm1f(d) - (double)d;
      }
      const double H = (double)p.ent[i];
      acc[0] += w * (double)s;
      acc[1] += w * H;
      acc[2] += w * kl;
      acc[3] += H;
      acc[4] += (double)rho;
      acc[5] += clipped ? 1.0 : 0.0;
      acc[6] += kl;
      acc[7] += w;
    }
  }
#pragma unroll
  for (int f = 0; f < kRollSums; ++f) acc[f] = wave_sum(acc[f]);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if (lane == 0)
#pragma unroll
    for (int f = 0; f < kRollSums; ++f) sh[wv][f] = acc[f];
  __syncthreads();
  if (threadIdx.x < kRollSums) {
    double t = 0.0;
    for (int k = 0; k < 4; ++k) t += sh[k][threadIdx.x];
    p.rsum[(int64_t)r * kRollSums + threadIdx.x] = t;
  }
}

__global__ void __launch_bounds__(1024) k_loss_final(LossParams p) {
  constexpr int NF = 7;   // J, J_pg, then the sums of H, rho, clipped, KL, w
  __shared__ double sh[16][NF];
  double a[NF] = {0, 0, 0, 0, 0, 0, 0};
  const double c = (double)p.ent_coef, beta = (double)p.kl_coef;
  for (int r = threadIdx.x; r < p.R; r += 1024) {
    const int q = p.gidx[r];
    const int n = p.rnpol[r];
    if (q < 0 || n == 0) continue;
    const double* rs = p.rsum + (int64_t)r * kRollSums;
    const double denom = p.agg == RLK_AGG_SEQ_MEAN_TOKEN_MEAN ? (double)n * (double)p.gsize[q] : 1.0;
    a[0] += (rs[0] + c * rs[1] - beta * rs[2]) / denom;
    a[1] += rs[0] / denom;
    a[2] += rs[3];
    a[3] += rs[4];
    a[4] += rs[5];
    a[5] += rs[6];
    a[6] += rs[7];
  }
#pragma unroll
  for (int f = 0; f < NF; ++f) a[f] = wave_sum(a[f]);
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  if (lane == 0)
#pragma unroll
    for (int f = 0; f < NF; ++f) sh[wv][f] = a[f];
  __syncthreads();
  if (threadIdx.x == 0) {
    double t[NF] = {0, 0, 0, 0, 0, 0, 0};
    for (int k = 0; k < 16; ++k)
      for (int f = 0; f < NF; ++f) t[f] += sh[k][f];
    const int n_eff = p.hdr->n_eff;
    const int Q = p.hdr->n_groups;
    double norm;
    if (p.agg == RLK_AGG_SEQ_MEAN_TOKEN_MEAN) norm = p.norm_override > 0 ? p.norm_override : (double)Q;
    else norm = p.norm_override > 0 ? p.norm_override : (double)n_eff;
    const bool empty = n_eff == 0 || Q == 0;
    const float loss = empty ? 0.0f : (float)(-t[0] / norm);
    const float pg = empty ? 0.0f : (float)(-t[1] / norm);
    if (p.loss) p.loss[0] = loss;
    if (p.stats) {
      rlk_pg_stats_t st;
      st.loss = loss;
      st.pg_loss = pg;
      st.entropy_mean = n_eff ? (float)(t[2] / n_eff) : 0.0f;
      st.ratio_mean = n_eff ? (float)(t[3] / n_eff) : 0.0f;
      st.clip_frac = n_eff ? (float)(t[4] / n_eff) : 0.0f;
      st.kl_mean = n_eff ? (float)(t[5] / n_eff) : 0.0f;
      st.tis_mean = n_eff ? (float)(t[6] / n_eff) : 1.0f;
      st.n_groups = Q;
      st.n_valid_rollouts = p.hdr->n_valid;
      st.n_policy_tokens = n_eff;
      st.n_chunks = p.nchunks;
      st.n_dz_chunks = p.hdr->n_dz_chunks;
      st.n_grad_tokens = p.hdr->n_grad;
      *p.stats = st;
    }
  }
}

// ---- rows that are not trained: dhidden row = 0 and the scattered per-token outputs = 0.
template <typename T>
__global__ void __launch_bounds__(256)
k_zero_fill(const uint8_t* keep, int64_t N, int d, T* dh, float* o1, float* o2, float* o3) {
  // keep 0: not trained (dh row and per-token outputs 0); 2: trained with a zero surrogate gradient
  // (dh row 0, per-token outputs kept); 1: trained
  const int64_t t = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (t >= N || keep[t] == 1) return;
  const int lane = threadIdx.x & 63;
  if (lane == 0 && keep[t] == 0) {
    if (o1) o1[t] = 0.0f;
    if (o2) o2[t] = 0.0f;
    if (o3) o3[t] = 0.0f;
  }
  if (!dh) return;
  constexpr int EPC = 16 / sizeof(T);
  const int nch = d / EPC;
  u32x4* row = reinterpret_cast<u32x4*>(dh + t * d);
  for (int c = lane; c < nch; c += 64) row[c] = u32x4{0, 0, 0, 0};
}

}  // namespace

hipError_t launch_transpose_w(int dtype, const void* W, void* WT, int V, int64_t Vp, int d, int64_t ldw,
                              hipStream_t s) {
  dim3 grid((unsigned)(Vp / 64), (unsigned)((d + 63) / 64));
  prof_mark(KK_TRANSPOSE_W, true, s);
  if (dtype == RLK_DTYPE_BF16)
    k_transpose_w<uint16_t><<<grid, 256, 0, s>>>((const uint16_t*)W, (uint16_t*)WT, V, Vp, d, ldw);
  else
    k_transpose_w<float><<<grid, 256, 0, s>>>((const float*)W, (float*)WT, V, Vp, d, ldw);
  prof_mark(KK_TRANSPOSE_W, false, s);
  return hipGetLastError();
}

hipError_t launch_gather(int dtype, const void* hidden, int d, const int32_t* idx, const WsHeader* hdr, int64_t c0,
                         int64_t Mc, void* hc, void* ht, int64_t ldt, bool want_ht, hipStream_t s) {
  dim3 grid((unsigned)((Mc + 63) / 64), (unsigned)((d + 63) / 64));
  prof_mark(KK_GATHER, true, s);
  if (dtype == RLK_DTYPE_BF16)
    k_gather<uint16_t><<<grid, 256, 0, s>>>((const uint16_t*)hidden, d, idx, hdr, c0, Mc, (uint16_t*)hc,
                                            (uint16_t*)ht, ldt, want_ht ? 1 : 0);
  else
    k_gather<float><<<grid, 256, 0, s>>>((const float*)hidden, d, idx, hdr, c0, Mc, (float*)hc, (float*)ht, ldt,
                                         want_ht ? 1 : 0);
  prof_mark(KK_GATHER, false, s);
  return hipGetLastError();
}

hipError_t launch_target_logit(const void* hc, int d, const void* W, const int32_t* ytgt, const WsHeader* hdr,
                               int64_t c0, int64_t Mc, int V, float inv_tau, float* zr, int32_t* fb,
                               hipStream_t s) {
  prof_mark(KK_TARGET_LOGIT, true, s);
  k_target_logit<<<(unsigned)((Mc + 3) / 4), 256, 0, s>>>((const uint16_t*)hc, d, (const uint16_t*)W, ytgt, hdr, c0,
                                                          Mc, V, inv_tau, zr, fb);
  prof_mark(KK_TARGET_LOGIT, false, s);
  return hipGetLastError();
}

hipError_t launch_hidden_t(const void* hc, int d, const float* st, const int32_t* fb, const WsHeader* hdr,
                           int64_t c0, int64_t Mc, void* ht, int64_t ldt, hipStream_t s) {
  dim3 grid((unsigned)((Mc + 63) / 64), (unsigned)((d + 63) / 64));
  prof_mark(KK_HIDDEN_T, true, s);
  k_hidden_t<<<grid, 256, 0, s>>>((const uint16_t*)hc, d, st, fb, hdr, c0, Mc, (uint16_t*)ht, ldt);
  prof_mark(KK_HIDDEN_T, false, s);
  return hipGetLastError();
}

hipError_t launch_combine(const TokenParams& p, hipStream_t s) {
  prof_mark(KK_COMBINE, true, s);
  k_combine<<<(unsigned)((p.Mc + 63) / 64), 256, 0, s>>>(p);
  prof_mark(KK_COMBINE, false, s);
  return hipGetLastError();
}

hipError_t launch_dz(int dtype, const DzParams& p, hipStream_t s) {
  const int64_t nvt = p.Vp / kVocabTile, ntb = (p.Mc + 63) / 64;
  prof_mark(KK_DZ, true, s);
  if (p.fb) {
    const unsigned grid = (unsigned)std::min<int64_t>(nvt * ntb, kDzBlocks);
    if (dtype == RLK_DTYPE_BF16) k_dz_flagged<uint16_t><<<grid, 256, 0, s>>>(p);
    else k_dz_flagged<float><<<grid, 256, 0, s>>>(p);
  } else {
    const dim3 grid((unsigned)nvt, (unsigned)ntb);
    if (dtype == RLK_DTYPE_BF16) {
      if (p.has_ent) k_dz<uint16_t, true><<<grid, 256, 0, s>>>(p);
      else k_dz<uint16_t, false><<<grid, 256, 0, s>>>(p);
    } else {
      if (p.has_ent) k_dz<float, true><<<grid, 256, 0, s>>>(p);
      else k_dz<float, false><<<grid, 256, 0, s>>>(p);
    }
  }
  prof_mark(KK_DZ, false, s);
  return hipGetLastError();
}

hipError_t launch_loss(const LossParams& p, hipStream_t s, int) {
  if (p.R > 0) {
    prof_mark(KK_LOSS_ROLLOUT, true, s);
    k_loss_rollout<<<p.R, 256, 0, s>>>(p);
    prof_mark(KK_LOSS_ROLLOUT, false, s);
  }
  prof_mark(KK_LOSS_FINAL, true, s);
  k_loss_final<<<1, 1024, 0, s>>>(p);
  prof_mark(KK_LOSS_FINAL, false, s);
  return hipGetLastError();
}

hipError_t launch_zero_fill(int dtype, const uint8_t* keep, int64_t N, int d, void* dh, float* o1, float* o2,
                            float* o3, hipStream_t s) {
  if (N <= 0) return hipSuccess;
  prof_mark(KK_ZERO_FILL, true, s);
  const unsigned blocks = (unsigned)((N + 3) / 4);
  if (dtype == RLK_DTYPE_BF16)
    k_zero_fill<uint16_t><<<blocks, 256, 0, s>>>(keep, N, d, (uint16_t*)dh, o1, o2, o3);
  else
    k_zero_fill<float><<<blocks, 256, 0, s>>>(keep, N, d, (float*)dh, o1, o2, o3);
  prof_mark(KK_ZERO_FILL, false, s);
  return hipGetLastError();
}

}  // namespace rlk
