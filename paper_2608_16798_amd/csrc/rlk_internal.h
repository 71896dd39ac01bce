// Internal declarations shared by the HIP translation units of librlk.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/rlk.h"

namespace rlk {

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Storage type of a bf16 element (bit pattern).
struct bf16_t {
  uint16_t bits;
};

// Tile geometry of the MFMA GEMMs (see k_gemm.hip).
constexpr int kTile = 256;       // BM = BN = 256
constexpr int kVocabTile = 256;  // vocabulary rows per forward tile = per online-LSE partial
constexpr int kChunkAlign = 256; // chunk_rows granularity
constexpr int kKAlign = 64;      // K padding of the chunk buffers (bf16 elements per stage)
constexpr int kGemmSliceBytes = 128;  // bytes of K per GEMM pipeline slice and row

// Token-reference layout of the stored probabilities (bf16 fwd+bwd without an entropy term):
// q_tj = exp(z_tj - ref_t) with ref_t = the target logit z_{t,y_t}, the same for every vocabulary
// tile of the token, so dL/dz = diag(s) q up to the target entry (s_t = -g_t exp(ref_t - lse_t)).
// A tile whose maximum exceeds ref_t by more than kRefSpan stores against max - kRefSpan instead
// and marks the chunk, whose dz is then formed explicitly; kRefQMax and kRefSMin bound the patched
// target entry and |s_t| for the same purpose (no bf16 overflow, no fp32 denormal scales).
constexpr float kRefSpan = 40.0f;
constexpr float kRefQMax = 1e30f;
constexpr float kRefSMin = 1e-30f;

// Split-K plan of a gradient GEMM with at most mmax x n outputs and kbytes of K per row: with
// fewer than 128 output tiles the K range is split over s workgroups per tile (each at least 4
// slices), so the launch still fills the GPU; the fp32 partials go to a workspace buffer of
// s x (rows rounded to 256) x (n rounded to 256) and a reduction kernel adds them in split order.
struct SplitK {
  int s;        // splits (1 = none)
  int kslices;  // K slices per split
};
inline SplitK splitk_plan(int64_t mmax, int64_t n, int64_t kbytes) {
  const int64_t tiles = ((mmax + kTile - 1) / kTile) * ((n + kTile - 1) / kTile);
  const int64_t nk = (kbytes + kGemmSliceBytes - 1) / kGemmSliceBytes;
  SplitK p = {1, (int)(nk > 0 ? nk : 1)};
  if (tiles <= 0 || tiles >= 128) return p;
  int64_t s = 512 / tiles;
  if (s > nk / 4) s = nk / 4;
  if (s > 64) s = 64;
  if (s < 2) return p;
  const int64_t ks = (nk + s - 1) / s;
  p.s = (int)((nk + ks - 1) / ks);
  p.kslices = (int)ks;
  if (p.s < 2) p = {1, (int)nk};
  return p;
}
inline size_t splitk_bytes(int64_t mmax, int64_t n, const SplitK& p) {
  if (p.s < 2) return 0;
  return (size_t)p.s * (size_t)((mmax + kTile - 1) / kTile * kTile) * (size_t)((n + kTile - 1) / kTile * kTile) * 4;
}
constexpr int kScanTile = 4096;  // tokens per compaction block
constexpr int kMaxRollouts = 16384;
constexpr int kRollSums = 8;     // per-rollout fp64 sums of the loss reduction

enum KernelKind {
  KK_BEGIN = 0,
  KK_COUNT,
  KK_SCAN,
  KK_WRITE_IDX,
  KK_ROLLOUT_OFFSETS,
  KK_GROUP_RANK,
  KK_GROUP_STATS,
  KK_ADVANTAGE,
  KK_TRANSPOSE_W,
  KK_GATHER,
  KK_FWD_GEMM,
  KK_COMBINE,
  KK_DZ,
  KK_DH_GEMM,
  KK_DW_GEMM,
  KK_LOSS_ROLLOUT,
  KK_LOSS_FINAL,
  KK_ZERO_FILL,
  KK_GAE,
  KK_VALUE_LOSS,
  KK_VALUE_HEAD,
  KK_TARGET_LOGIT,
  KK_HIDDEN_T,
  KK_COUNT_KINDS
};

// Device-side header at offset 0 of every workspace.
struct WsHeader {
  int32_t status;    // RLK_DERR_* bits
  int32_t n_eff;     // number of trained tokens
  int32_t n_groups;  // Q
  int32_t n_valid;   // non-excluded rollouts
  int32_t n_grad;    // leading trained tokens of the compacted list that carry a surrogate gradient
  int32_t ref_fallback;  // current chunk: 1 = its token-reference layout does not hold, dz explicit
  int32_t n_dz_chunks;   // chunks whose dz was formed explicitly
  int32_t pad[57];
};

// Byte offsets of the workspace segments (all 256-aligned).
struct WsLayout {
  size_t total = 0;
  size_t hdr = 0;
  // token arrays [N]
  size_t keep = 0, idx = 0, tokr = 0, ytgt = 0, zy = 0, lse = 0, logp = 0, ent = 0, gt = 0, et = 0;
  // compaction block scan [nblk]
  size_t blkcnt = 0, blkoff = 0;
  // rollouts [R]
  size_t rstart = 0, rnpol = 0, members = 0, gstart = 0, gidx = 0, gsize = 0, gmu = 0, gsig = 0, geq = 0, adv = 0;
  size_t rsum = 0;  // double [R][kRollSums]
  // chunk buffers
  size_t pm = 0, ps = 0, pu = 0;   // float [nvt][Mc]
  size_t hc = 0;                   // T [Mc][d]
  size_t ht = 0;                   // T [d][Mc]
  size_t q = 0;                    // T [Mc][ldq]
  size_t dzt = 0;                  // T [Vp][ldt]
  size_t wt = 0;                   // T [d][ldw]
  size_t zr = 0, st = 0;           // float [Mc]: reference logit and dz row scale per chunk row
  size_t part = 0;                 // float split-K partials of the dhidden / dW GEMMs (0 = none)
  SplitK sk_dh = {1, 1}, sk_dw = {1, 1};
  // dW launch of a large shape (sk_dw none): output tiles from row dw_m0 on (the partial last wave of
  // 256 tiles, whole tile rows) go to a second launch split over K by sk_dwt; dw_m0 = 0: one launch
  int64_t dw_m0 = 0;
  SplitK sk_dwt = {1, 1};
  int64_t rows_bound = 0;          // trained tokens the chunk loop covers (N, or the caller's bound)
  // chunk c < n1 covers [c Mc1, min((c + 1) Mc1, g_rows)); the others [g_rows + (c - n1) Mc2, + Mc2)
  // (without a hint: n1 = nchunks, Mc1 = Mc2 = Mc, g_rows = nchunks Mc)
  int64_t Mc1 = 0, Mc2 = 0, g_rows = 0;
  int32_t n1 = 0;
  int64_t Mc = 0;                  // chunk rows
  int64_t Vp = 0;                  // vocabulary padded to 256
  // Row strides (elements) of the chunk buffers read by the gradient GEMMs: padded by 64 when the
  // byte stride would be a multiple of 2 KiB (such strides were measured up to 28 % slower)
  int64_t ldq = 0, ldt = 0, ldw = 0;
  int32_t nvt = 0;                 // vocabulary tiles
  int32_t nblk = 0;                // compaction blocks
  int32_t nchunks = 0;             // chunk iterations launched (ceil(N / Mc))
};

// ---- launchers (k_segment.hip) ----
hipError_t launch_begin(int32_t* status_hdr, const int32_t* cu, int R, int64_t N, hipStream_t s);
// zero_adv [R] (may be NULL): the rollouts' advantages; the tokens of a rollout whose advantage is
// exactly 0 are listed after all others (n_grad = the count before them; NULL: n_grad = n_eff).
hipError_t launch_compact(const uint8_t* mask, const int32_t* cu, const int32_t* gid, int R, int64_t N,
                          const int32_t* targets, int V, int32_t max_policy, const float* zero_adv, char* ws,
                          const WsLayout& L, hipStream_t s);
// members [R] (rollouts of the kept groups, group by group), gstart [R + 1] (run starts), gidx [R],
// and per group gsize, gmu, gsig, geq [R]; R <= kMaxRollouts.
hipError_t launch_advantage(int R, const float* rewards, const int32_t* gid, float adv_eps, int32_t* members,
                            int32_t* gstart, int32_t* gidx, int32_t* gsize, double* gmu, double* gsig, int32_t* geq,
                            float* adv, WsHeader* hdr, hipStream_t s);

// ---- launchers (k_token.hip) ----
hipError_t launch_transpose_w(int dtype, const void* W, void* WT, int V, int64_t Vp, int d, int64_t ldw,
                              hipStream_t s);
hipError_t launch_gather(int dtype, const void* hidden, int d, const int32_t* idx, const WsHeader* hdr,
                         int64_t c0, int64_t Mc, void* hc, void* ht, int64_t ldt, bool want_ht, hipStream_t s);
// bf16: zr[t] = (hc[t] . W[ytgt[c0 + t]]) / tau for the chunk's rows; clears *fb.
hipError_t launch_target_logit(const void* hc, int d, const void* W, const int32_t* ytgt, const WsHeader* hdr,
                               int64_t c0, int64_t Mc, int V, float inv_tau, float* zr, int32_t* fb,
                               hipStream_t s);
// bf16: HT[j][t] = hc[t][j] * (*fb ? 1 : st[t]) (zero columns t >= rows, up to the K pad).
hipError_t launch_hidden_t(const void* hc, int d, const float* st, const int32_t* fb, const WsHeader* hdr,
                           int64_t c0, int64_t Mc, void* ht, int64_t ldt, hipStream_t s);

struct TokenParams {
  const WsHeader* hdr;
  int64_t c0, Mc;
  int nvt;
  const float *pm, *ps, *pu, *zy;
  const int32_t *idx, *tokr, *ytgt;
  float *lse, *logp, *ent, *gt, *et;
  float *logp_out, *ent_out, *lse_out;   // scattered [N] outputs, may be null
  // loss terms (fwd+bwd only)
  int with_grad;
  const float* old_logp;
  const float* adv;
  const int32_t *rnpol, *gidx, *gsize;
  float eps_low, eps_high, ent_coef;
  int agg;
  double norm_override;
  const float* rollout_logp;   // truncated importance sampling (NULL = off)
  float tis_cap;
  const float* ref_logp;       // KL term (NULL = off)
  float kl_coef;
  const float* token_adv;      // per-token advantages (NULL = group advantages)
  float inv_tau;               // 1 / temperature: dL/d(W h) = dL/dz / tau
  // token-reference layout (bf16; zr = NULL: off): reference logits zr [Mc]; out: the target entries of
  // q [Mc][ldq] and q^T [Vp][ldqt], the row scales st [Mc] and *fb |= 1 where the bounds fail
  const float* zr;
  float* st;
  int32_t* fb;
  void *q, *qt;
  int64_t ldq, ldqt;
  int V;
};
hipError_t launch_combine(const TokenParams& p, hipStream_t s);

struct DzParams {
  const WsHeader* hdr;
  int64_t c0, Mc, Vp;
  int64_t ldq, ldt;   // row strides of q / dz and of dz^T (elements)
  int V;
  void* q;        // in: exp(z - m_tile) ; out: dz, [Mc][ldq] (columns < Vp)
  void* dzt;      // out: dz transposed, [Vp][ldt] (columns < Mc)
  const float *pm, *lse, *logp, *ent, *gt, *et;
  const int32_t* ytgt;
  int has_ent;
  const int32_t* fb;   // non-NULL: run only when *fb != 0 (token-reference layout not usable)
  int32_t* ndz;        // counts the chunks that ran (may be NULL)
};
hipError_t launch_dz(int dtype, const DzParams& p, hipStream_t s);

struct LossParams {
  const WsHeader* hdr;
  int R;
  const int32_t *rstart, *rnpol, *gidx, *gsize, *idx;
  const float *logp, *ent, *old_logp, *adv;
  double* rsum;
  float eps_low, eps_high, ent_coef;
  int agg;
  double norm_override;
  const float* rollout_logp;
  float tis_cap;
  const float* ref_logp;
  float kl_coef;
  const float* token_adv;
  float* loss;
  rlk_pg_stats_t* stats;
  int32_t nchunks;
};
hipError_t launch_loss(const LossParams& p, hipStream_t s, int prof_kind_first);

hipError_t launch_zero_fill(int dtype, const uint8_t* keep, int64_t N, int d, void* dh, float* o1, float* o2,
                            float* o3, hipStream_t s);

// ---- launchers (k_ppo.hip) ----
hipError_t launch_gae(int64_t N, int R, const int32_t* cu, const uint8_t* mask, const float* values,
                      const float* rewards, const int32_t* gid, float gamma, float lam, float* adv, float* ret,
                      hipStream_t s);
hipError_t launch_value_loss(int64_t N, int R, const int32_t* cu, const uint8_t* mask, const float* values,
                             const float* ret, const int32_t* gid, double* part, double* total, float* loss,
                             float* dv, hipStream_t s);

size_t value_head_workspace(int64_t N, int d);
hipError_t launch_value_head_fwd(int dtype, int64_t N, int d, int R, const void* h, const void* w, float b,
                                 const uint8_t* mask, const int32_t* cu, const int32_t* gid, float* values,
                                 hipStream_t s);
hipError_t launch_value_head_bwd(int dtype, int64_t N, int d, int R, const void* h, const void* w,
                                 const uint8_t* mask, const int32_t* cu, const int32_t* gid, const float* dv,
                                 void* dh, int accumulate, float* dw, float* dbias, char* ws, hipStream_t s);

// ---- launchers (k_gemm.hip) ----
struct GemmArgs {
  const void* A;
  const void* B;
  int64_t lda, ldb;      // elements
  int M, N, K;           // static maxima (the data-dependent one is derived on device)
  const WsHeader* hdr;   // n_eff
  int64_t c0;            // first compacted row of the chunk
  int64_t Mc;            // chunk capacity
  // forward epilogue
  const int32_t* ytgt;   // compacted targets
  float* zy;
  float *pm, *ps, *pu;   // [nvt][Mc]
  void* q;               // [Mc][ldq]
  int64_t ldq;
  int V;
  float inv_tau;         // logits z = acc / tau
  // token-reference layout (bf16 forward; zr = NULL: each tile stores against its own maximum):
  // reference logits zr [Mc], q^T [Vp][ldqt] written beside q, *fb = 1 where a tile clamps
  const float* zr;
  void* qt;
  int64_t ldqt;
  int32_t* fb;
  // dhidden epilogue
  void* out;
  const int32_t* idx;
  int64_t ldo;
  const float* rs;       // row scales [Mc] applied unless *rs_off != 0 (NULL: none)
  const int32_t* rs_off;
  // dW epilogue
  float* dw;
  int accumulate;
  // split K (dhidden and dW): ksplit workgroups per output tile, each over kslices slices, write
  // fp32 partials part[split][row][col] (row stride ldp, mp rows per split); a reduction kernel
  // then applies the epilogue
  int ksplit;
  int kslices;
  float* part;
  int64_t ldp;
  int64_t mp;
};
hipError_t launch_fwd_gemm(int dtype, const GemmArgs& a, bool store_q, hipStream_t s);
hipError_t launch_dh_gemm(int dtype, const GemmArgs& a, hipStream_t s);
hipError_t launch_dw_gemm(int dtype, const GemmArgs& a, hipStream_t s);

// ---- error reporting for host-side entry points in other files (rlk_api.hip) ----
rlk_status_t report_error(rlk_status_t code, const char* msg);

// ---- profiling (rlk_api.hip) ----
void prof_mark(int kind, bool begin, hipStream_t s);

}  // namespace rlk
