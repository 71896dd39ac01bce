// C-ABI entry points of librlk: argument validation, workspace layout, the chunk loop and
// the launch sequence of the hot path.  No device memory is allocated here; every buffer
// comes from the caller.
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <string>
#include <vector>

#include "rlk_internal.h"

namespace rlk {

// Layouts the Python binding mirrors.
static_assert(sizeof(rlk_batch_t) == 40, "rlk_batch_t layout");
static_assert(sizeof(rlk_pg_params_t) == 80, "rlk_pg_params_t layout");
static_assert(sizeof(rlk_pg_stats_t) == 64, "rlk_pg_stats_t layout");

namespace {

thread_local std::string g_last_error;

rlk_status_t fail(rlk_status_t code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
rlk_status_t fail(rlk_status_t code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

rlk_status_t hip_fail(hipError_t e, const char* what) {
  return fail(RLK_EHIP, "%s: %s", what, hipGetErrorString(e));
}

}  // namespace

rlk_status_t report_error(rlk_status_t code, const char* msg) { return fail(code, "%s", msg); }

namespace {

constexpr size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
// Row tensors (hidden, W, dhidden) are read and written with 16-byte vector accesses.
inline bool misaligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) != 0; }
inline int64_t roundup(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

struct Alloc {
  size_t off = 0;
  constexpr size_t take(size_t bytes) {
    size_t o = off;
    off = align256(off + bytes);
    return o;
  }
};

bool debug_sync() {
  static const bool v = [] {
    const char* e = getenv("RLK_DEBUG_SYNC");
    return e && e[0] && e[0] != '0';
  }();
  return v;
}

rlk_status_t check_batch(const rlk_batch_t* b) {
  if (!b) return fail(RLK_EINVAL, "batch descriptor is NULL");
  if (b->dtype != RLK_DTYPE_F32 && b->dtype != RLK_DTYPE_BF16) return fail(RLK_EDTYPE, "unknown dtype %d", b->dtype);
  if (b->N < 0 || b->R < 0) return fail(RLK_ESHAPE, "negative N (%lld) or R (%d)", (long long)b->N, b->R);
  if (b->N >= ((int64_t)1 << 31)) return fail(RLK_ESHAPE, "N = %lld exceeds the int32 token index", (long long)b->N);
  if (b->R == 0 && b->N != 0) return fail(RLK_ESHAPE, "R = 0 with N = %lld tokens", (long long)b->N);
  if (b->R > kMaxRollouts) return fail(RLK_ESHAPE, "R = %d exceeds the supported %d rollouts", b->R, kMaxRollouts);
  if (b->d < 8 || b->d % 8 != 0) return fail(RLK_ESHAPE, "d = %d must be a positive multiple of 8", b->d);
  if (b->d > RLK_MAX_DIM) return fail(RLK_ESHAPE, "d = %d exceeds %d", b->d, RLK_MAX_DIM);
  if (b->V < 1 || b->V > RLK_MAX_DIM) return fail(RLK_ESHAPE, "V = %d must lie in [1, %d]", b->V, RLK_MAX_DIM);
  if (b->R > 0 && !b->cu_seqlens) return fail(RLK_EINVAL, "cu_seqlens is NULL");
  if (b->temperature != 0.0f && !(b->temperature > 0.0f && isfinite(b->temperature)))
    return fail(RLK_EINVAL, "temperature must be 0 (= 1) or finite and > 0");
  if (b->max_policy_tokens < 0) return fail(RLK_EINVAL, "max_policy_tokens must be >= 0");
  return RLK_OK;
}

// Row stride (elements) of a chunk buffer with rows of x elements of esz bytes: x rounded up to 64,
// plus 64 more when the byte stride would be a multiple of 2 KiB.  Operand row strides with a
// power-of-two factor of 2 KiB or more made the gradient GEMMs 4-28 % slower in measurements;
// smaller factors (the qwen8b shapes) are left alone, where padding measured no better.
int64_t pad_ld(int64_t x, int64_t esz) {
  int64_t r = (x + 63) / 64 * 64;
  if ((r * esz) % 2048 == 0) r += 64;
  return r;
}

// split-K arguments of a gradient GEMM (rows of the partial buffer padded to whole tiles)
void set_split(GemmArgs& g, const SplitK& p, char* part) {
  g.ksplit = p.s;
  g.kslices = p.kslices;
  if (p.s > 1) {
    g.part = reinterpret_cast<float*>(part);
    g.ldp = (int64_t)(g.N + kTile - 1) / kTile * kTile;
    g.mp = (int64_t)(g.M + kTile - 1) / kTile * kTile;
  }
}

// 1 / tau of the batch's logits (z = W h / tau)
float inv_temperature(const rlk_batch_t* b) { return b->temperature == 0.0f ? 1.0f : 1.0f / b->temperature; }

// Rows per chunk for a batch known to hold at most B trained tokens, with at most cap rows per chunk:
// the fewest chunks, and among the row counts giving that many, the one whose chunks fill the most
// whole waves of 256 output tiles in the forward and dhidden GEMMs (the dW GEMM's tile count does
// not depend on the chunk rows); ties go to the smaller workspace.
int64_t plan_chunk_rows(int64_t B, int64_t cap, int64_t d, int64_t Vp) {
  const int64_t nch = (B + cap - 1) / cap;
  const int64_t rmin = roundup((B + nch - 1) / nch, kChunkAlign);
  const int64_t tv = Vp / kTile, td = (d + kTile - 1) / kTile;
  auto waves = [](int64_t tiles) { return (tiles + 255) / 256; };
  int64_t best = rmin, best_cost = -1;
  for (int64_t r = rmin; r <= cap; r += kChunkAlign) {
    int64_t cost = 0, left = B;
    for (int64_t c = 0; c < nch && left > 0; ++c) {
      const int64_t rows = std::min(r, left), tc = (rows + kTile - 1) / kTile;
      cost += waves(tv * tc) * d + waves(tc * td) * Vp;
      left -= rows;
    }
    if (left > 0) continue;  // r too small for nch chunks
    if (best_cost < 0 || cost < best_cost) {
      best = r;
      best_cost = cost;
    }
  }
  return best;
}

// The dW GEMM's V x d outputs form whole waves of 256 tiles plus a partial last wave, whose time is
// that of a whole one (K = the chunk's tokens, the longest tiles of the step at large chunks).  The
// tile rows of that wave go to a second launch split over K into as many parts as fit one wave
// (partials reduced in split order), when that is at least 2 parts.
void plan_dw_tail(int64_t V, int64_t d, int64_t kbytes, WsLayout& L) {
  L.dw_m0 = 0;
  L.sk_dwt = {1, 1};
  if (L.sk_dw.s > 1) return;
  const int64_t tm = (V + kTile - 1) / kTile, tn = (d + kTile - 1) / kTile, tail = tm * tn % 256;
  if (tail == 0) return;
  const int64_t r = (tail + tn - 1) / tn;  // tile rows holding the partial wave
  const int64_t s = 256 / (r * tn);
  const int64_t nk = (kbytes + kGemmSliceBytes - 1) / kGemmSliceBytes;
  if (r >= tm || s < 2 || nk < 2) return;
  const int64_t ks = (nk + s - 1) / s;
  L.sk_dwt = {(int)((nk + ks - 1) / ks), (int)ks};
  if (L.sk_dwt.s < 2) {
    L.sk_dwt = {1, 1};
    return;
  }
  L.dw_m0 = (tm - r) * kTile;
}

// The dhidden GEMM of a chunk known to hold at most `rows` trained tokens (the caller's bound): its
// tile rows x d output tiles end in a partial wave of 256 tiles that costs a whole wave of the longest
// tiles of the step (K = Vp).  Those tile rows go to a second launch split over K into s parts, which
// takes ceil(tail tiles x s / 256) waves of 1/s of the work; s (2-16, each part at least 4 slices) is
// the smallest within 0.02 waves of the quickest, and only a saving of a tenth of a wave is taken.
struct DhTail {
  int64_t m0 = 0;  // first tile row of the tail (rows); 0 = one launch
  SplitK sk = {1, 1};
  int64_t rows = 0;  // rows of the tail launch (whole tiles)
};
DhTail plan_dh_tail(int64_t rows, int64_t d, int64_t kbytes) {
  DhTail t;
  const int64_t tc = (rows + kTile - 1) / kTile, tn = (d + kTile - 1) / kTile, tail = tc * tn % 256;
  const int64_t nk = (kbytes + kGemmSliceBytes - 1) / kGemmSliceBytes;
  if (tail == 0 || tc * tn < 256) return t;
  const int64_t r = (tail + tn - 1) / tn;
  if (r >= tc) return t;
  auto waves = [&](int64_t s) { return (double)((r * tn * s + 255) / 256) / (double)s; };
  double best = 1.0;
  for (int64_t s = 2; s <= 16 && nk / s >= 4; ++s) best = std::min(best, waves(s));
  if (best > 0.9) return t;
  int64_t sel = 2;
  while (waves(sel) > best + 0.02) ++sel;
  const int64_t ks = (nk + sel - 1) / sel;
  const SplitK sk = {(int)((nk + ks - 1) / ks), (int)ks};
  if (sk.s < 2) return t;
  t.sk = sk;
  t.m0 = (tc - r) * kTile;
  t.rows = r * kTile;
  return t;
}

// Chunk c of the loop: first compacted row and capacity (rows the chunk's kernels may cover).
struct ChunkSpan {
  int64_t c0, rows;
};
ChunkSpan chunk_span(const WsLayout& L, int c) {
  if (c < L.n1) {
    const int64_t c0 = (int64_t)c * L.Mc1;
    return {c0, c0 < L.g_rows ? std::min(L.Mc1, L.g_rows - c0) : L.Mc1};
  }
  return {L.g_rows + (int64_t)(c - L.n1) * L.Mc2, L.Mc2};
}

// The caller's count of tokens with a possible surrogate gradient, when the backward skips the others.
int64_t grad_hint(const rlk_pg_params_t* p) {
  if (!p || p->grad_tokens <= 0) return 0;
  return p->entropy_coef == 0.0f && p->kl_coef == 0.0f && !p->token_adv ? p->grad_tokens : 0;
}

rlk_status_t layout(const rlk_batch_t* b, bool bwd, int64_t chunk_rows, int64_t grad_tokens, WsLayout& L) {
  const int64_t esz = b->dtype == RLK_DTYPE_BF16 ? 2 : 4;
  const int64_t N = b->N, R = b->R, d = b->d, V = b->V;
  L.Vp = roundup(V, kVocabTile);
  L.nvt = (int32_t)(L.Vp / kVocabTile);
  L.nblk = (int32_t)((N + kScanTile - 1) / kScanTile);
  if (L.nblk < 1) L.nblk = 1;
  if (chunk_rows < 0 || chunk_rows % kChunkAlign != 0 || chunk_rows > RLK_MAX_CHUNK_ROWS)
    return fail(RLK_ESHAPE, "chunk_rows = %lld must be a multiple of %d in [0, %d]", (long long)chunk_rows,
                kChunkAlign, RLK_MAX_CHUNK_ROWS);
  int64_t Mc = chunk_rows;
  if (Mc == 0) {
    int64_t per_row = (int64_t)L.nvt * 12 + d * esz;
    if (bwd) per_row += d * esz + 2 * L.Vp * esz;
    const int64_t budget = bwd ? ((int64_t)40 << 30) : ((int64_t)4 << 30);
    Mc = budget / per_row / kChunkAlign * kChunkAlign;
    if (Mc > 65536) Mc = 65536;
    if (Mc < kChunkAlign) Mc = kChunkAlign;
    const int64_t cap = roundup(N > 0 ? N : 1, kChunkAlign);
    if (Mc > cap) Mc = cap;
  }
  // rows the chunk loop has to cover: all N, or the caller's bound on the trained tokens
  const int64_t B = b->max_policy_tokens > 0 ? std::min<int64_t>(b->max_policy_tokens, N) : N;
  const int64_t cap = Mc;
  if (b->max_policy_tokens > 0 && B > 0) Mc = plan_chunk_rows(B, cap, d, L.Vp);
  L.Mc = Mc;
  L.rows_bound = B;
  L.nchunks = (int32_t)((B + Mc - 1) / Mc);
  if (bwd && L.nchunks < 1) L.nchunks = 1;
  L.n1 = L.nchunks;
  L.Mc1 = L.Mc2 = Mc;
  L.g_rows = (int64_t)L.nchunks * Mc;  // every chunk Mc rows wide (row strides stay multiples of 256)
  const int64_t G = grad_tokens > 0 && grad_tokens < B ? roundup(grad_tokens, kChunkAlign) : 0;
  if (bwd && b->max_policy_tokens > 0 && G > 0 && G < B) {
    // the tokens with a gradient come first in the compacted list: chunks planned over them, then
    // over the rest (whose backward kernels, when the hint is right, find no rows and return; a
    // wrong hint only moves work between chunks, since the kernels read the counts from the device).
    // The boundary is rounded up to
    // whole 256-row tiles, which keeps every chunk's rows, and so the row stride of its online-LSE
    // partials, a multiple of 256.
    L.Mc1 = plan_chunk_rows(G, cap, d, L.Vp);
    L.Mc2 = plan_chunk_rows(B - G, cap, d, L.Vp);
    L.n1 = (int32_t)((G + L.Mc1 - 1) / L.Mc1);
    L.g_rows = G;
    L.nchunks = L.n1 + (int32_t)((B - G + L.Mc2 - 1) / L.Mc2);
    L.Mc = Mc = std::max(L.Mc1, L.Mc2);
  }

  Alloc a;
  L.hdr = a.take(sizeof(WsHeader));
  L.keep = a.take((size_t)N);
  L.blkcnt = a.take((size_t)L.nblk * 8);  // two halves: tokens with and without a surrogate gradient
  L.blkoff = a.take((size_t)L.nblk * 8);
  L.idx = a.take((size_t)N * 4);
  L.tokr = a.take((size_t)N * 4);
  L.ytgt = a.take((size_t)N * 4);
  L.zy = a.take((size_t)N * 4);
  L.lse = a.take((size_t)N * 4);
  L.logp = a.take((size_t)N * 4);
  L.ent = a.take((size_t)N * 4);
  L.gt = a.take((size_t)N * 4);
  L.et = a.take((size_t)N * 4);
  L.rstart = a.take((size_t)R * 4);
  L.rnpol = a.take((size_t)R * 4);
  L.members = a.take((size_t)R * 4);
  L.gstart = a.take((size_t)(R + 1) * 4);
  L.gidx = a.take((size_t)R * 4);
  L.gsize = a.take((size_t)R * 4);
  L.gmu = a.take((size_t)R * 8);
  L.gsig = a.take((size_t)R * 8);
  L.geq = a.take((size_t)R * 4);
  L.adv = a.take((size_t)R * 4);
  L.rsum = a.take((size_t)R * 8 * kRollSums);
  L.pm = a.take((size_t)L.nvt * Mc * 4);
  L.ps = a.take((size_t)L.nvt * Mc * 4);
  L.pu = a.take((size_t)L.nvt * Mc * 4);
  L.hc = a.take((size_t)(Mc * d * esz));
  if (bwd) {
    L.ldq = pad_ld(L.Vp, esz);
    L.ldt = pad_ld(Mc, esz);
    L.ldw = pad_ld(L.Vp, esz);
    L.ht = a.take((size_t)(d * L.ldt * esz));
    L.q = a.take((size_t)(Mc * L.ldq * esz));
    L.dzt = a.take((size_t)(L.Vp * L.ldt * esz));
    L.wt = a.take((size_t)(d * L.ldw * esz));
    L.zr = a.take((size_t)Mc * 4);
    L.st = a.take((size_t)Mc * 4);
    // split-K partials of the dhidden and dW GEMMs (used one after the other)
    L.sk_dh = splitk_plan(Mc, d, L.Vp * esz);
    L.sk_dw = splitk_plan(V, d, Mc * esz);
    plan_dw_tail(V, d, Mc * esz, L);
    size_t pb = std::max({splitk_bytes(Mc, d, L.sk_dh), splitk_bytes(V, d, L.sk_dw),
                          splitk_bytes(V - L.dw_m0, d, L.sk_dwt)});
    if (L.sk_dh.s == 1 && b->max_policy_tokens > 0)
      for (int c = 0; c < L.nchunks; ++c) {
        const ChunkSpan cs = chunk_span(L, c);
        if (cs.c0 >= B) break;
        const DhTail t = plan_dh_tail(std::min(cs.rows, B - cs.c0), d, L.Vp * esz);
        if (t.m0 > 0) pb = std::max(pb, splitk_bytes(t.rows, d, t.sk));
      }
    if (pb > 0) L.part = a.take(pb);
  }
  // The GEMMs address each 256-row operand panel with 32-bit buffer offsets and mark rows past a
  // ragged panel with the offset 0x80000000: every panel must span at most 2 GiB.
  const int64_t lds[] = {d, L.ldq, L.ldt, L.ldw};
  for (int64_t ld : lds)
    if ((int64_t)kTile * ld * esz > ((int64_t)1 << 31))
      return fail(RLK_ESHAPE, "a %d-row operand panel of row stride %lld exceeds 2 GiB", kTile, (long long)ld);
  L.total = a.off;
  return RLK_OK;
}

constexpr size_t advantage_ws_bytes(int32_t R) {
  Alloc a;
  a.take(sizeof(WsHeader));
  a.take((size_t)R * 4);        // members
  a.take((size_t)(R + 1) * 4);  // run starts
  a.take((size_t)R * 4);  // gidx
  a.take((size_t)R * 4);  // gsize
  a.take((size_t)R * 8);  // mu
  a.take((size_t)R * 8);  // sigma
  a.take((size_t)R * 4);  // all-equal flags
  return a.off;
}

rlk_status_t check_ws(const void* ws, size_t have, size_t need) {
  if (!ws) return fail(RLK_EWORKSPACE, "workspace is NULL");
  if (reinterpret_cast<uintptr_t>(ws) % 256 != 0) return fail(RLK_EWORKSPACE, "workspace must be 256-byte aligned");
  if (have < need)
    return fail(RLK_EWORKSPACE, "workspace has %zu bytes, %zu needed", have, need);
  return RLK_OK;
}

rlk_status_t finish(hipError_t e, const char* what, const void* ws, hipStream_t s) {
  if (e != hipSuccess) return hip_fail(e, what);
  if (debug_sync()) {
    hipError_t e2 = hipStreamSynchronize(s);
    if (e2 != hipSuccess) return hip_fail(e2, "hipStreamSynchronize");
    int32_t st = 0;
    e2 = hipMemcpy(&st, ws, sizeof(int32_t), hipMemcpyDeviceToHost);
    if (e2 != hipSuccess) return hip_fail(e2, "hipMemcpy(status)");
    if (st != 0) return fail(RLK_EDATA, "device data error flags 0x%x", st);
  }
  return RLK_OK;
}

#define RLK_TRY(expr, what)                      \
  do {                                           \
    hipError_t _e = (expr);                      \
    if (_e != hipSuccess) return hip_fail(_e, what); \
  } while (0)

// ---------------------------------------------------------------- profiling
struct ProfRec {
  int kind;
  hipEvent_t a, b;
};
// Events are created when profiling begins (a pool reused across profiling windows), so a launch
// inside the window only records two events and takes no allocation.
struct Prof {
  std::mutex mu;
  bool on = false;
  std::vector<ProfRec> recs;
  std::vector<hipEvent_t> pool;  // created events
  size_t next = 0;               // first pool event not recorded in this window
  hipEvent_t open = nullptr;
  int open_kind = -1;
  hipEvent_t take() {
    if (next == pool.size()) {
      hipEvent_t ev;
      if (hipEventCreate(&ev) != hipSuccess) return nullptr;
      pool.push_back(ev);
    }
    return pool[next++];
  }
};
constexpr size_t kProfPoolEvents = 8192;
Prof& prof() {
  static Prof p;
  return p;
}

const char* kKindNames[KK_COUNT_KINDS] = {
    "begin",        "compact_count", "compact_scan",  "compact_write", "rollout_offsets", "group_rank",
    "group_stats",  "advantage",     "transpose_w",   "gather",        "fwd_lse_gemm",    "lse_combine",
    "dz",           "dh_gemm",       "dw_gemm",       "loss_rollout",  "loss_final",      "zero_fill",
    "gae",          "value_loss",    "value_head",    "target_logit",  "hidden_t"};

}  // namespace

void prof_mark(int kind, bool begin, hipStream_t s) {
  Prof& P = prof();
  if (!P.on) return;
  std::lock_guard<std::mutex> lk(P.mu);
  if (begin) {
    hipEvent_t ev = P.take();
    if (!ev) return;
    (void)hipEventRecord(ev, s);
    P.open = ev;
    P.open_kind = kind;
  } else if (P.open && P.open_kind == kind) {
    hipEvent_t ev = P.take();
    if (!ev) return;
    (void)hipEventRecord(ev, s);
    P.recs.push_back({kind, P.open, ev});
    P.open = nullptr;
    P.open_kind = -1;
  }
}

namespace {

rlk_status_t check_advantage_args(int32_t R, const float* rewards, const int32_t* group_ids, float adv_eps,
                                  const float* adv) {
  if (R < 0 || R > kMaxRollouts) return fail(RLK_ESHAPE, "R = %d outside [0, %d]", R, kMaxRollouts);
  if (R > 0 && (!rewards || !group_ids || !adv)) return fail(RLK_EINVAL, "rewards, group_ids or adv is NULL");
  if (!(adv_eps >= 0.0f) || !isfinite(adv_eps)) return fail(RLK_EINVAL, "adv_eps must be finite and >= 0");
  return RLK_OK;
}

// The launches of rlk_group_advantage on a validated workspace of advantage_ws_bytes(R) bytes.
rlk_status_t advantage_call(int32_t R, const float* rewards, const int32_t* group_ids, float adv_eps, float* adv,
                            int32_t* group_index, int32_t* n_groups, void* ws, void* stream) {
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  Alloc a;
  char* w = static_cast<char*>(ws);
  WsHeader* hdr = reinterpret_cast<WsHeader*>(w + a.take(sizeof(WsHeader)));
  int32_t* members = reinterpret_cast<int32_t*>(w + a.take((size_t)R * 4));
  int32_t* gstart = reinterpret_cast<int32_t*>(w + a.take((size_t)(R + 1) * 4));
  int32_t* gidx_ws = reinterpret_cast<int32_t*>(w + a.take((size_t)R * 4));
  int32_t* gsize = reinterpret_cast<int32_t*>(w + a.take((size_t)R * 4));
  double* gmu = reinterpret_cast<double*>(w + a.take((size_t)R * 8));
  double* gsig = reinterpret_cast<double*>(w + a.take((size_t)R * 8));
  int32_t* geq = reinterpret_cast<int32_t*>(w + a.take((size_t)R * 4));
  int32_t* gidx = group_index ? group_index : gidx_ws;
  RLK_TRY(launch_begin(reinterpret_cast<int32_t*>(hdr), nullptr, 0, 0, s), "begin");
  RLK_TRY(launch_advantage(R, rewards, group_ids, adv_eps, members, gstart, gidx, gsize, gmu, gsig, geq, adv, hdr, s),
          "advantage");
  if (n_groups)
    RLK_TRY(hipMemcpyAsync(n_groups, &hdr->n_groups, sizeof(int32_t), hipMemcpyDeviceToDevice, s), "copy n_groups");
  return finish(hipSuccess, "", ws, s);
}

// ---------------------------------------------------------------- fixed device scratch
// Workspace of rlk_group_advantage_noalloc: the advantage workspace of the largest supported rollout
// count, one copy per device, held by every GPU the library runs on until the process ends.  On the
// host, `scratch` names a host-side stand-in, never the device memory: host code only uses the
// device address that hipGetSymbolAddress returns for the current device, looked up once per device.
constexpr size_t kAdvScratchBytes = advantage_ws_bytes(kMaxRollouts);
static_assert(kAdvScratchBytes == 590336, "the size stated in rlk.h");
static __device__ __align__(256) char scratch[kAdvScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of `scratch` on the device of `stream`, which must be the current device.
rlk_status_t device_scratch(void* stream, void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (stream) {
    hipDevice_t sdev = 0;
    e = hipStreamGetDevice(reinterpret_cast<hipStream_t>(stream), &sdev);
    if (e != hipSuccess) return hip_fail(e, "hipStreamGetDevice");
    if ((int)sdev != dev) return fail(RLK_EINVAL, "the stream belongs to device %d, the current device is %d", (int)sdev, dev);
  }
  if (dev < 0 || dev >= kMaxDevices) return fail(RLK_EINVAL, "device %d outside [0, %d)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (!p || (reinterpret_cast<uintptr_t>(p) & 255) != 0) return fail(RLK_EHIP, "scratch address is not 256-aligned");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return RLK_OK;
}

}  // namespace

}  // namespace rlk

using namespace rlk;

extern "C" {

rlk_status_t rlk_workspace_size(const rlk_batch_t* b, const rlk_pg_params_t* p, size_t* bytes) {
  if (!bytes) return fail(RLK_EINVAL, "bytes is NULL");
  rlk_status_t st = check_batch(b);
  if (st) return st;
  WsLayout L;
  st = layout(b, p != nullptr, p ? p->chunk_rows : 0, grad_hint(p), L);
  if (st) return st;
  *bytes = L.total;
  return RLK_OK;
}

rlk_status_t rlk_advantage_workspace_size(int32_t R, size_t* bytes) {
  if (!bytes) return fail(RLK_EINVAL, "bytes is NULL");
  if (R < 0 || R > kMaxRollouts) return fail(RLK_ESHAPE, "R = %d outside [0, %d]", R, kMaxRollouts);
  *bytes = advantage_ws_bytes(R);
  return RLK_OK;
}

rlk_status_t rlk_logprob_fwd(const rlk_batch_t* b, const void* hidden, const void* W, const int32_t* targets,
                             const uint8_t* mask, float* logp, float* entropy, float* lse, void* ws,
                             size_t ws_bytes, void* stream) {
  rlk_status_t st = check_batch(b);
  if (st) return st;
  if (b->N > 0 && (!hidden || !targets || !logp)) return fail(RLK_EINVAL, "hidden, targets or logp is NULL");
  if (!W) return fail(RLK_EINVAL, "W is NULL");
  if (misaligned16(hidden) || misaligned16(W)) return fail(RLK_EINVAL, "hidden and W must be 16-byte aligned");
  WsLayout L;
  st = layout(b, false, 0, 0, L);
  if (st) return st;
  st = check_ws(ws, ws_bytes, L.total);
  if (st) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  WsHeader* hdr = reinterpret_cast<WsHeader*>(w + L.hdr);
  const int64_t N = b->N;

  RLK_TRY(launch_begin(reinterpret_cast<int32_t*>(hdr), b->cu_seqlens, b->R, N, s), "begin");
  if (N == 0) return finish(hipSuccess, "", ws, s);
  RLK_TRY(launch_compact(mask, b->cu_seqlens, nullptr, b->R, N, targets, b->V, b->max_policy_tokens, nullptr, w, L,
                         s),
          "compact");
  for (int c = 0; c < L.nchunks; ++c) {
    const int64_t c0 = (int64_t)c * L.Mc;
    RLK_TRY(launch_gather(b->dtype, hidden, b->d, reinterpret_cast<const int32_t*>(w + L.idx), hdr, c0, L.Mc,
                          w + L.hc, nullptr, 0, false, s),
            "gather");
    GemmArgs g = {};
    g.A = W;
    g.B = w + L.hc;
    g.lda = b->d;
    g.ldb = b->d;
    g.M = b->V;
    g.N = (int)L.Mc;
    g.K = b->d;
    g.hdr = hdr;
    g.c0 = c0;
    g.Mc = L.Mc;
    g.ytgt = reinterpret_cast<const int32_t*>(w + L.ytgt);
    g.zy = reinterpret_cast<float*>(w + L.zy);
    g.pm = reinterpret_cast<float*>(w + L.pm);
    g.ps = reinterpret_cast<float*>(w + L.ps);
    g.pu = reinterpret_cast<float*>(w + L.pu);
    g.V = b->V;
    g.inv_tau = inv_temperature(b);
    RLK_TRY(launch_fwd_gemm(b->dtype, g, false, s), "fwd_gemm");
    TokenParams tp = {};
    tp.inv_tau = inv_temperature(b);
    tp.hdr = hdr;
    tp.c0 = c0;
    tp.Mc = L.Mc;
    tp.nvt = L.nvt;
    tp.pm = g.pm;
    tp.ps = g.ps;
    tp.pu = g.pu;
    tp.zy = g.zy;
    tp.idx = reinterpret_cast<const int32_t*>(w + L.idx);
    tp.tokr = reinterpret_cast<const int32_t*>(w + L.tokr);
    tp.ytgt = g.ytgt;
    tp.lse = reinterpret_cast<float*>(w + L.lse);
    tp.logp = reinterpret_cast<float*>(w + L.logp);
    tp.ent = reinterpret_cast<float*>(w + L.ent);
    tp.gt = reinterpret_cast<float*>(w + L.gt);
    tp.et = reinterpret_cast<float*>(w + L.et);
    tp.logp_out = logp;
    tp.ent_out = entropy;
    tp.lse_out = lse;
    tp.with_grad = 0;
    RLK_TRY(launch_combine(tp, s), "combine");
  }
  RLK_TRY(launch_zero_fill(b->dtype, reinterpret_cast<const uint8_t*>(w + L.keep), N, b->d, nullptr, logp, entropy,
                           lse, s),
          "zero_fill");
  return finish(hipSuccess, "", ws, s);
}

rlk_status_t rlk_compact(const rlk_batch_t* b, const uint8_t* mask, const int32_t* group_ids,
                         const int32_t* targets, int32_t* idx, int32_t* tok_rollout, int32_t* n_pol, int32_t* n_eff,
                         void* ws, size_t ws_bytes, void* stream) {
  rlk_status_t st = check_batch(b);
  if (st) return st;
  if (!n_eff || (b->N > 0 && (!idx || !tok_rollout)) || (b->R > 0 && !n_pol))
    return fail(RLK_EINVAL, "idx, tok_rollout, n_pol or n_eff is NULL");
  WsLayout L;
  st = layout(b, false, 0, 0, L);
  if (st) return st;
  st = check_ws(ws, ws_bytes, L.total);
  if (st) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  WsHeader* hdr = reinterpret_cast<WsHeader*>(w + L.hdr);
  RLK_TRY(launch_begin(reinterpret_cast<int32_t*>(hdr), b->cu_seqlens, b->R, b->N, s), "begin");
  RLK_TRY(launch_compact(mask, b->cu_seqlens, group_ids, b->R, b->N, targets, b->V, b->max_policy_tokens, nullptr,
                         w, L, s),
          "compact");
  if (b->N > 0) {
    RLK_TRY(hipMemcpyAsync(idx, w + L.idx, (size_t)b->N * 4, hipMemcpyDeviceToDevice, s), "copy idx");
    RLK_TRY(hipMemcpyAsync(tok_rollout, w + L.tokr, (size_t)b->N * 4, hipMemcpyDeviceToDevice, s), "copy tok_rollout");
  }
  if (b->R > 0)
    RLK_TRY(hipMemcpyAsync(n_pol, w + L.rnpol, (size_t)b->R * 4, hipMemcpyDeviceToDevice, s), "copy n_pol");
  RLK_TRY(hipMemcpyAsync(n_eff, &hdr->n_eff, 4, hipMemcpyDeviceToDevice, s), "copy n_eff");
  return finish(hipSuccess, "", ws, s);
}

rlk_status_t rlk_group_advantage(int32_t R, const float* rewards, const int32_t* group_ids, float adv_eps,
                                 float* adv, int32_t* group_index, int32_t* n_groups, void* ws, size_t ws_bytes,
                                 void* stream) {
  rlk_status_t st = check_advantage_args(R, rewards, group_ids, adv_eps, adv);
  if (st) return st;
  st = check_ws(ws, ws_bytes, advantage_ws_bytes(R));
  if (st) return st;
  return advantage_call(R, rewards, group_ids, adv_eps, adv, group_index, n_groups, ws, stream);
}

rlk_status_t rlk_group_advantage_noalloc(int32_t R, const float* rewards, const int32_t* group_ids, float adv_eps,
                                         float* adv, int32_t* group_index, int32_t* n_groups, void* stream) {
  rlk_status_t st = check_advantage_args(R, rewards, group_ids, adv_eps, adv);
  if (st) return st;
  if (advantage_ws_bytes(R) > kAdvScratchBytes)
    return fail(RLK_ESHAPE, "R = %d needs %zu bytes of scratch, the fixed array holds %zu", R, advantage_ws_bytes(R),
                kAdvScratchBytes);
  void* ws = nullptr;
  st = device_scratch(stream, &ws);
  if (st) return st;
  return advantage_call(R, rewards, group_ids, adv_eps, adv, group_index, n_groups, ws, stream);
}

rlk_status_t rlk_pg_loss_fwd_bwd(const rlk_batch_t* b, const void* hidden, const void* W, const int32_t* targets,
                                 const uint8_t* mask, const float* old_logp, const float* rewards,
                                 const int32_t* group_ids, const rlk_pg_params_t* p, float* loss, void* dhidden,
                                 float* dW, float* logp_out, float* entropy_out, rlk_pg_stats_t* stats, void* ws,
                                 size_t ws_bytes, void* stream) {
  rlk_status_t st = check_batch(b);
  if (st) return st;
  if (!p) return fail(RLK_EINVAL, "params is NULL");
  if (!W || !dW || !loss) return fail(RLK_EINVAL, "W, dW or loss is NULL");
  if (b->N > 0 && (!hidden || !targets || !old_logp || !dhidden))
    return fail(RLK_EINVAL, "hidden, targets, old_logp or dhidden is NULL");
  if (misaligned16(hidden) || misaligned16(W) || misaligned16(dhidden))
    return fail(RLK_EINVAL, "hidden, W and dhidden must be 16-byte aligned");
  if (b->R > 0 && (!rewards || !group_ids)) return fail(RLK_EINVAL, "rewards or group_ids is NULL");
  if (!(p->eps_low >= 0.0f && p->eps_low < 1.0f) || !(p->eps_high >= 0.0f) || !isfinite(p->eps_high))
    return fail(RLK_EINVAL, "clip range must satisfy 0 <= eps_low < 1 and finite eps_high >= 0");
  if (!(p->adv_eps >= 0.0f) || !isfinite(p->adv_eps)) return fail(RLK_EINVAL, "adv_eps must be finite and >= 0");
  if (!isfinite(p->entropy_coef)) return fail(RLK_EINVAL, "entropy_coef must be finite");
  if (p->agg != RLK_AGG_SEQ_MEAN_TOKEN_MEAN && p->agg != RLK_AGG_TOKEN_MEAN)
    return fail(RLK_EINVAL, "unknown aggregation %d", p->agg);
  if (p->accumulate_dW != 0 && p->accumulate_dW != 1) return fail(RLK_EINVAL, "accumulate_dW must be 0 or 1");
  if (!(p->norm_override >= 0.0) || !isfinite(p->norm_override))
    return fail(RLK_EINVAL, "norm_override must be finite and >= 0");
  if (p->rollout_logp ? !(p->tis_cap > 0.0f && isfinite(p->tis_cap)) : p->tis_cap != 0.0f)
    return fail(RLK_EINVAL, "tis_cap must be finite and > 0 with rollout_logp, and 0 without");
  if (!(p->kl_coef >= 0.0f) || !isfinite(p->kl_coef)) return fail(RLK_EINVAL, "kl_coef must be finite and >= 0");
  if (p->kl_coef > 0.0f && !p->ref_logp) return fail(RLK_EINVAL, "kl_coef > 0 needs ref_logp");
  WsLayout L;
  if (p->grad_tokens < 0) return fail(RLK_EINVAL, "grad_tokens must be >= 0");
  st = layout(b, true, p->chunk_rows, grad_hint(p), L);
  if (st) return st;
  st = check_ws(ws, ws_bytes, L.total);
  if (st) return st;

  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  char* w = static_cast<char*>(ws);
  WsHeader* hdr = reinterpret_cast<WsHeader*>(w + L.hdr);
  const int64_t N = b->N;
  const int R = b->R;
  auto F = [&](size_t off) { return reinterpret_cast<float*>(w + off); };
  auto I = [&](size_t off) { return reinterpret_cast<int32_t*>(w + off); };

  RLK_TRY(launch_begin(reinterpret_cast<int32_t*>(hdr), b->cu_seqlens, R, N, s), "begin");
  RLK_TRY(launch_advantage(R, rewards, group_ids, p->adv_eps, I(L.members), I(L.gstart), I(L.gidx), I(L.gsize),
                           reinterpret_cast<double*>(w + L.gmu), reinterpret_cast<double*>(w + L.gsig), I(L.geq),
                           F(L.adv), hdr, s),
          "advantage");
  // With the advantage-weighted surrogate as the only term (no entropy bonus, KL term or per-token
  // advantages), a rollout of advantage exactly 0 has an exactly zero gradient: its tokens go last in
  // the compacted list and the backward covers the tokens before them.
  const bool zero_grad_skip = p->entropy_coef == 0.0f && p->kl_coef == 0.0f && !p->token_adv;
  RLK_TRY(launch_compact(mask, b->cu_seqlens, group_ids, R, N, targets, b->V, b->max_policy_tokens,
                         zero_grad_skip ? F(L.adv) : nullptr, w, L, s),
          "compact");
  RLK_TRY(launch_transpose_w(b->dtype, W, w + L.wt, b->V, L.Vp, b->d, L.ldw, s), "transpose_w");
  // Token-reference layout (bf16 without an entropy term): the forward stores q against each token's
  // target logit and writes q^T as well; the combine makes dz = diag(s) q exact, the dhidden GEMM and
  // the scaled transpose of the gathered rows apply s, and the explicit dz pass runs only for chunks
  // flagged on the device (a token whose target lies too far below its largest logits).
  const bool ref_layout = b->dtype == RLK_DTYPE_BF16 && p->entropy_coef == 0.0f;
  const size_t esz = b->dtype == RLK_DTYPE_BF16 ? 2 : 4;
  int32_t* fb = &hdr->ref_fallback;
  for (int c = 0; c < L.nchunks; ++c) {
    const ChunkSpan cs = chunk_span(L, c);
    const int64_t c0 = cs.c0, Mcc = cs.rows;
    RLK_TRY(launch_gather(b->dtype, hidden, b->d, I(L.idx), hdr, c0, Mcc, w + L.hc, w + L.ht, L.ldt, !ref_layout,
                          s),
            "gather");
    if (ref_layout)
      RLK_TRY(launch_target_logit(w + L.hc, b->d, W, I(L.ytgt), hdr, c0, Mcc, b->V, inv_temperature(b), F(L.zr),
                                  fb, s),
              "target_logit");
    GemmArgs g = {};
    g.A = W;
    g.B = w + L.hc;
    g.lda = b->d;
    g.ldb = b->d;
    g.M = b->V;
    g.N = (int)Mcc;
    g.K = b->d;
    g.hdr = hdr;
    g.c0 = c0;
    g.Mc = Mcc;
    g.ytgt = I(L.ytgt);
    g.zy = F(L.zy);
    g.pm = F(L.pm);
    g.ps = F(L.ps);
    g.pu = F(L.pu);
    g.q = w + L.q;
    g.ldq = L.ldq;
    g.V = b->V;
    g.inv_tau = inv_temperature(b);
    if (ref_layout) {
      g.zr = F(L.zr);
      g.qt = w + L.dzt;
      g.ldqt = L.ldt;
      g.fb = fb;
    }
    RLK_TRY(launch_fwd_gemm(b->dtype, g, true, s), "fwd_gemm");

    TokenParams tp = {};
    tp.inv_tau = inv_temperature(b);
    tp.hdr = hdr;
    tp.c0 = c0;
    tp.Mc = Mcc;
    tp.nvt = L.nvt;
    tp.pm = g.pm;
    tp.ps = g.ps;
    tp.pu = g.pu;
    tp.zy = g.zy;
    tp.idx = I(L.idx);
    tp.tokr = I(L.tokr);
    tp.ytgt = I(L.ytgt);
    tp.lse = F(L.lse);
    tp.logp = F(L.logp);
    tp.ent = F(L.ent);
    tp.gt = F(L.gt);
    tp.et = F(L.et);
    tp.logp_out = logp_out;
    tp.ent_out = entropy_out;
    tp.with_grad = 1;
    tp.old_logp = old_logp;
    tp.adv = F(L.adv);
    tp.rnpol = I(L.rnpol);
    tp.gidx = I(L.gidx);
    tp.gsize = I(L.gsize);
    tp.eps_low = p->eps_low;
    tp.eps_high = p->eps_high;
    tp.ent_coef = p->entropy_coef;
    tp.agg = p->agg;
    tp.norm_override = p->norm_override;
    tp.rollout_logp = p->rollout_logp;
    tp.tis_cap = p->tis_cap;
    tp.ref_logp = p->kl_coef > 0.0f ? p->ref_logp : nullptr;
    tp.kl_coef = p->kl_coef;
    tp.token_adv = p->token_adv;
    if (ref_layout) {
      tp.zr = F(L.zr);
      tp.st = F(L.st);
      tp.fb = fb;
      tp.q = w + L.q;
      tp.qt = w + L.dzt;
      tp.ldq = L.ldq;
      tp.ldqt = L.ldt;
      tp.V = b->V;
    }
    RLK_TRY(launch_combine(tp, s), "combine");

    DzParams dp = {};
    dp.hdr = hdr;
    dp.c0 = c0;
    dp.Mc = Mcc;
    dp.Vp = L.Vp;
    dp.ldq = L.ldq;
    dp.ldt = L.ldt;
    dp.V = b->V;
    dp.q = w + L.q;
    dp.dzt = w + L.dzt;
    dp.pm = g.pm;
    dp.lse = tp.lse;
    dp.logp = tp.logp;
    dp.ent = tp.ent;
    dp.gt = tp.gt;
    dp.et = tp.et;
    dp.ytgt = tp.ytgt;
    dp.has_ent = p->entropy_coef != 0.0f;
    dp.fb = ref_layout ? fb : nullptr;
    dp.ndz = &hdr->n_dz_chunks;
    RLK_TRY(launch_dz(b->dtype, dp, s), "dz");
    if (ref_layout)
      RLK_TRY(launch_hidden_t(w + L.hc, b->d, F(L.st), fb, hdr, c0, Mcc, w + L.ht, L.ldt, s), "hidden_t");

    GemmArgs h = {};
    h.A = w + L.q;
    h.B = w + L.wt;
    h.lda = L.ldq;
    h.ldb = L.ldw;
    h.M = (int)Mcc;
    h.N = b->d;
    h.K = (int)L.Vp;
    h.hdr = hdr;
    h.c0 = c0;
    h.Mc = Mcc;
    h.out = dhidden;
    h.idx = I(L.idx);
    h.ldo = b->d;
    if (ref_layout) {
      h.rs = F(L.st);
      h.rs_off = fb;
    }
    set_split(h, L.sk_dh, w + L.part);
    const DhTail dt = L.sk_dh.s == 1 && b->max_policy_tokens > 0
                          ? plan_dh_tail(std::min(Mcc, L.rows_bound - c0), b->d, L.Vp * esz)
                          : DhTail{};
    if (dt.m0 > 0) {
      // the tile rows of the partial last wave, split over K: the same GEMM on the chunk rows from
      // c0 + m0 (the kernels read the trained-token count relative to c0)
      GemmArgs t = h;
      t.A = w + L.q + (size_t)dt.m0 * L.ldq * esz;
      t.M = (int)dt.rows;
      t.c0 = c0 + dt.m0;
      t.Mc = std::min(dt.rows, Mcc - dt.m0);  // a ragged chunk ends inside the last tile row
      if (t.rs) t.rs += dt.m0;
      set_split(t, dt.sk, w + L.part);
      h.M = (int)dt.m0;
      h.Mc = dt.m0;
      RLK_TRY(launch_dh_gemm(b->dtype, h, s), "dh_gemm");
      RLK_TRY(launch_dh_gemm(b->dtype, t, s), "dh_gemm tail");
    } else {
      RLK_TRY(launch_dh_gemm(b->dtype, h, s), "dh_gemm");
    }

    GemmArgs k = {};
    k.A = w + L.dzt;
    k.B = w + L.ht;
    k.lda = L.ldt;
    k.ldb = L.ldt;
    k.M = b->V;
    k.N = b->d;
    k.K = (int)Mcc;
    k.hdr = hdr;
    k.c0 = c0;
    k.Mc = Mcc;
    k.dw = dW;
    k.ldo = b->d;
    k.accumulate = p->accumulate_dW;
    set_split(k, L.sk_dw, w + L.part);
    if (L.dw_m0 > 0) {
      // the tile rows of the partial last wave, split over K
      GemmArgs t = k;
      t.A = w + L.dzt + (size_t)L.dw_m0 * L.ldt * esz;
      t.M = b->V - (int)L.dw_m0;
      t.dw = dW + L.dw_m0 * b->d;
      set_split(t, L.sk_dwt, w + L.part);
      k.M = (int)L.dw_m0;
      RLK_TRY(launch_dw_gemm(b->dtype, k, s), "dw_gemm");
      RLK_TRY(launch_dw_gemm(b->dtype, t, s), "dw_gemm tail");
    } else {
      RLK_TRY(launch_dw_gemm(b->dtype, k, s), "dw_gemm");
    }
  }

  LossParams lp = {};
  lp.hdr = hdr;
  lp.R = R;
  lp.rstart = I(L.rstart);
  lp.rnpol = I(L.rnpol);
  lp.gidx = I(L.gidx);
  lp.gsize = I(L.gsize);
  lp.idx = I(L.idx);
  lp.logp = F(L.logp);
  lp.ent = F(L.ent);
  lp.old_logp = old_logp;
  lp.adv = F(L.adv);
  lp.rsum = reinterpret_cast<double*>(w + L.rsum);
  lp.eps_low = p->eps_low;
  lp.eps_high = p->eps_high;
  lp.ent_coef = p->entropy_coef;
  lp.agg = p->agg;
  lp.norm_override = p->norm_override;
  lp.rollout_logp = p->rollout_logp;
  lp.tis_cap = p->tis_cap;
  lp.ref_logp = p->kl_coef > 0.0f ? p->ref_logp : nullptr;
  lp.kl_coef = p->kl_coef;
  lp.token_adv = p->token_adv;
  lp.loss = loss;
  lp.stats = stats;
  lp.nchunks = L.nchunks;
  RLK_TRY(launch_loss(lp, s, 0), "loss");
  RLK_TRY(launch_zero_fill(b->dtype, reinterpret_cast<const uint8_t*>(w + L.keep), N, b->d, dhidden, logp_out,
                           entropy_out, nullptr, s),
          "zero_fill");
  return finish(hipSuccess, "", ws, s);
}

rlk_status_t rlk_gae(int64_t N, int32_t R, const int32_t* cu_seqlens, const uint8_t* mask, const float* values,
                     const float* rewards, const int32_t* group_ids, float gamma, float lam, float* adv,
                     float* returns, void* stream) {
  if (N < 0 || R < 0 || R > kMaxRollouts) return fail(RLK_ESHAPE, "N = %lld or R = %d out of range", (long long)N, R);
  if (!(gamma >= 0.0f && gamma <= 1.0f) || !(lam >= 0.0f && lam <= 1.0f))
    return fail(RLK_EINVAL, "gamma and lam must lie in [0, 1]");
  if (R == 0) return RLK_OK;
  if (!cu_seqlens || !rewards) return fail(RLK_EINVAL, "cu_seqlens or rewards is NULL");
  if (N > 0 && (!mask || !values || !adv)) return fail(RLK_EINVAL, "mask, values or adv is NULL");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  RLK_TRY(launch_gae(N, R, cu_seqlens, mask, values, rewards, group_ids, gamma, lam, adv, returns, s), "gae");
  return RLK_OK;
}

rlk_status_t rlk_value_workspace_size(int32_t R, size_t* bytes) {
  if (!bytes) return fail(RLK_EINVAL, "bytes is NULL");
  if (R < 0 || R > kMaxRollouts) return fail(RLK_ESHAPE, "R = %d outside [0, %d]", R, kMaxRollouts);
  Alloc a;
  a.take(sizeof(WsHeader));
  a.take(sizeof(double) * 2);
  a.take((size_t)R * 16);
  *bytes = a.off;
  return RLK_OK;
}

rlk_status_t rlk_value_loss(int64_t N, int32_t R, const int32_t* cu_seqlens, const uint8_t* mask,
                            const float* values, const float* returns, const int32_t* group_ids, float* loss,
                            float* dvalues, void* ws, size_t ws_bytes, void* stream) {
  if (N < 0 || R < 0 || R > kMaxRollouts) return fail(RLK_ESHAPE, "N = %lld or R = %d out of range", (long long)N, R);
  if (!loss) return fail(RLK_EINVAL, "loss is NULL");
  if (R > 0 && !cu_seqlens) return fail(RLK_EINVAL, "cu_seqlens is NULL");
  if (N > 0 && (!mask || !values || !returns)) return fail(RLK_EINVAL, "mask, values or returns is NULL");
  size_t need = 0;
  rlk_status_t st = rlk_value_workspace_size(R, &need);
  if (st) return st;
  st = check_ws(ws, ws_bytes, need);
  if (st) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  Alloc a;
  char* w = static_cast<char*>(ws);
  a.take(sizeof(WsHeader));
  double* total = reinterpret_cast<double*>(w + a.take(sizeof(double) * 2));
  double* part = reinterpret_cast<double*>(w + a.take((size_t)R * 16));
  RLK_TRY(launch_value_loss(N, R, cu_seqlens, mask, values, returns, group_ids, part, total, loss, dvalues, s),
          "value_loss");
  return RLK_OK;
}

rlk_status_t rlk_value_head_workspace_size(const rlk_batch_t* b, size_t* bytes) {
  if (!bytes) return fail(RLK_EINVAL, "bytes is NULL");
  rlk_status_t st = check_batch(b);
  if (st) return st;
  *bytes = value_head_workspace(b->N, b->d);
  return RLK_OK;
}

rlk_status_t rlk_value_head_fwd(const rlk_batch_t* b, const void* hidden, const void* w_v, float b_v,
                                const uint8_t* mask, const int32_t* group_ids, float* values, void* stream) {
  rlk_status_t st = check_batch(b);
  if (st) return st;
  if (!isfinite(b_v)) return fail(RLK_EINVAL, "b_v must be finite");
  if (b->N > 0 && (!hidden || !w_v || !values)) return fail(RLK_EINVAL, "hidden, w_v or values is NULL");
  if (misaligned16(hidden)) return fail(RLK_EINVAL, "hidden must be 16-byte aligned");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  RLK_TRY(launch_value_head_fwd(b->dtype, b->N, b->d, b->R, hidden, w_v, b_v, mask, b->cu_seqlens, group_ids,
                                values, s),
          "value_head_fwd");
  return RLK_OK;
}

rlk_status_t rlk_value_head_bwd(const rlk_batch_t* b, const void* hidden, const void* w_v, const uint8_t* mask,
                                const int32_t* group_ids, const float* dvalues, void* dhidden, int32_t accumulate,
                                float* dw_v, float* db_v, void* ws, size_t ws_bytes, void* stream) {
  rlk_status_t st = check_batch(b);
  if (st) return st;
  if (accumulate != 0 && accumulate != 1) return fail(RLK_EINVAL, "accumulate must be 0 or 1");
  if (!dw_v || !db_v) return fail(RLK_EINVAL, "dw_v or db_v is NULL");
  if (b->N > 0 && (!hidden || !w_v || !dvalues)) return fail(RLK_EINVAL, "hidden, w_v or dvalues is NULL");
  if (misaligned16(hidden) || misaligned16(dhidden))
    return fail(RLK_EINVAL, "hidden and dhidden must be 16-byte aligned");
  st = check_ws(ws, ws_bytes, value_head_workspace(b->N, b->d));
  if (st) return st;
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  RLK_TRY(launch_value_head_bwd(b->dtype, b->N, b->d, b->R, hidden, w_v, mask, b->cu_seqlens, group_ids, dvalues,
                                dhidden, accumulate, dw_v, db_v, static_cast<char*>(ws), s),
          "value_head_bwd");
  return RLK_OK;
}

rlk_status_t rlk_check_status(const void* ws, void* stream, int32_t* flags) {
  if (!ws) return fail(RLK_EINVAL, "workspace is NULL");
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  RLK_TRY(hipStreamSynchronize(s), "hipStreamSynchronize");
  int32_t st = 0;
  RLK_TRY(hipMemcpy(&st, ws, sizeof(int32_t), hipMemcpyDeviceToHost), "hipMemcpy(status)");
  if (flags) *flags = st;
  if (st != 0) return fail(RLK_EDATA, "device data error flags 0x%x", st);
  return RLK_OK;
}

const char* rlk_status_string(rlk_status_t s) {
  switch (s) {
    case RLK_OK: return "ok";
    case RLK_EINVAL: return "invalid argument";
    case RLK_ESHAPE: return "unsupported or inconsistent shape";
    case RLK_EDTYPE: return "unknown dtype";
    case RLK_EWORKSPACE: return "workspace missing, misaligned or too small";
    case RLK_EHIP: return "HIP runtime error";
    case RLK_EDATA: return "device data error";
    default: return "unknown status";
  }
}

const char* rlk_last_error(void) { return g_last_error.c_str(); }

int32_t rlk_version(void) { return RLK_VERSION; }

rlk_status_t rlk_profile_begin(void) {
  Prof& P = prof();
  std::lock_guard<std::mutex> lk(P.mu);
  P.recs.clear();
  P.next = 0;
  P.open = nullptr;
  P.open_kind = -1;
  while (P.pool.size() < kProfPoolEvents) {
    hipEvent_t ev;
    if (hipEventCreate(&ev) != hipSuccess) return fail(RLK_EHIP, "hipEventCreate failed");
    P.pool.push_back(ev);
  }
  P.on = true;
  return RLK_OK;
}

rlk_status_t rlk_profile_end(int32_t max_kinds, double* total_ms, int32_t* launches, int32_t* n_kinds) {
  Prof& P = prof();
  std::lock_guard<std::mutex> lk(P.mu);
  P.on = false;
  if (n_kinds) *n_kinds = KK_COUNT_KINDS;
  for (int k = 0; k < max_kinds && k < KK_COUNT_KINDS; ++k) {
    if (total_ms) total_ms[k] = 0.0;
    if (launches) launches[k] = 0;
  }
  rlk_status_t rc = RLK_OK;
  for (auto& r : P.recs) {
    float ms = 0.0f;
    if (hipEventSynchronize(r.b) != hipSuccess || hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) {
      rc = fail(RLK_EHIP, "event timing failed");
    } else if (r.kind < max_kinds) {
      if (total_ms) total_ms[r.kind] += ms;
      if (launches) launches[r.kind] += 1;
    }
  }
  P.recs.clear();
  P.next = 0;  // the events go back to the pool
  return rc;
}

const char* rlk_kernel_kind_name(int32_t kind) {
  if (kind < 0 || kind >= KK_COUNT_KINDS) return "";
  return kKindNames[kind];
}

}  // extern "C"
