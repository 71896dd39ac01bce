// MFMA GEMMs of the LM-head projection and its two gradient contractions, with fused
// epilogues.  One core computes C[m][n] = sum_k A[m][k] * B[n][k] with both operands
// K-contiguous ("NT"); the three uses are
//   forward : A = W [V, d],          B = gathered hidden [tokens, d]   -> online log-softmax
//   dhidden : A = dz [tokens, Vp],   B = W^T [d, Vp]                   -> scatter to dh[idx]
//   dW      : A = dz^T [Vp, tokens], B = hidden^T [d, tokens]          -> fp32 dW (+)=
// In the token-reference layout (dz = diag(s) q) the gradient GEMMs read the forward's q and q^T
// as A, the dhidden epilogue scales its rows by s and the dW GEMM's B is (diag(s) hidden)^T.
//
// Tile geometry (gfx950): a 256 x 256 output tile per workgroup of WAVES_M x WAVES_N = 2 x 4
// wavefronts (two per SIMD), each owning a 128 x 64 block of 32 x 32 v_mfma_f32_32x32x16_bf16
// tiles (fp32 operands use v_mfma_f32_32x32x2_f32) with its 128 fp32 accumulators per lane in
// the unified register file.  Operands stream through LDS in K slices of KS bytes per row,
// copied straight from global memory by buffer_load ... lds (no staging registers) into NSTAGE
// buffers; rows are XOR-swizzled at 16-byte granularity so MFMA fragment reads are bank-conflict
// free.  Each lane's MFMA fragment carries 8
// consecutive K elements of one row (16 bytes); A and B use the same K assignment, so the lane
// split of K inside the MFMA is irrelevant to the sum.
//
// The gradient GEMMs of shapes with few output tiles split K over several workgroups per tile
// (fp32 partials in the workspace, summed in split order by k_splitk_reduce).
//
// Output layout of a 32x32 MFMA block: lane l holds column (l % 32); accumulator register r
// holds row 8*(r/4) + 4*(l/32) + (r%4).  With vocabulary on M and tokens on N, every lane's
// accumulators belong to a single token, so the vocabulary reduction of the online
// log-softmax is in-register, then one cross-half exchange, then one LDS exchange between
// the wavefronts of a column.
#include "rlk_internal.h"

#include <algorithm>

namespace rlk {

namespace {

#ifndef RLK_KS
#define RLK_KS 128
#endif
#ifndef RLK_NSTAGE
#define RLK_NSTAGE 2
#endif
#ifndef RLK_WAVES_N
#define RLK_WAVES_N 4
#endif
constexpr int WAVES_M = 2;
constexpr int WAVES_N = RLK_WAVES_N;    // 2: one wavefront per SIMD; 4: two per SIMD
constexpr int NWAVE = WAVES_M * WAVES_N;
constexpr int NT = 64 * NWAVE;
constexpr int WTM = kTile / WAVES_M;    // rows of a wavefront's block
constexpr int WTN = kTile / WAVES_N;    // columns of a wavefront's block
constexpr int MBW = WTM / 32;           // 32x32 MFMA tiles per wavefront along M
constexpr int NBW = WTN / 32;           // ... along N
constexpr int KS = RLK_KS;              // bytes of K per pipeline slice per row (kGemmSliceBytes)
constexpr int NSTAGE = RLK_NSTAGE;      // LDS buffers in the copy pipeline
constexpr int CPR = KS / 16;            // 16-byte chunks per row of a slice
constexpr int RPI = 64 / CPR;           // rows per LDS-DMA instruction
constexpr int IPW = kTile / RPI / NWAVE;  // LDS-DMA instructions per wavefront per operand
constexpr int NKK = KS / 32;            // MFMA K steps per slice
constexpr int DMA_PER_SLICE = 2 * IPW;  // vector-memory instructions per wavefront per slice
constexpr int OPND_B = kTile * KS;      // one operand's slice
constexpr int STAGE_B = 2 * OPND_B;     // A + B
constexpr int PIPE_B = NSTAGE * STAGE_B;
static_assert(PIPE_B <= 131072 && KS == kGemmSliceBytes && IPW >= 1, "pipeline geometry");
constexpr int QROW = kTile * 2 + 16;    // LDS row stride of the bf16 probability tile (bytes)
constexpr int RED_OFF = kTile * QROW;   // 135168: reduction scratch after the staged tile
// The staged tile holds token t's 16-byte vocabulary chunk c at chunk c ^ qswz(t) of row t, so that
// the transposing reads of 8 tokens 8 apart (same chunk) fall in distinct bank groups.
__device__ __forceinline__ int qswz(int t) { return (t >> 3) & 7; }
constexpr int LDS_B = RED_OFF + 3 * WAVES_M * kTile * 4;  // >= PIPE_B
constexpr int GROUP_M = 16;
constexpr float kLog2e = 1.4426950408889634f;
constexpr int kBufferFlags = 0x00020000;  // raw buffer: 32-bit data format, offset range-checked

#define LDSP(p) ((__attribute__((address_space(3))) void*)(p))

// Scheduling hints for one MFMA K step: interleave the LDS fragment reads (and the global->LDS
// copies of the next slice) with the MFMA chain.
template <int NMFMA, int NDS, int NVMEM>
__device__ __forceinline__ void sched_step() {
#pragma unroll
  for (int i = 0; i < NMFMA; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
    if constexpr (NVMEM > 0) {
      if (i * NVMEM / NMFMA != (i + 1) * NVMEM / NMFMA) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      if ((i + 1) * NVMEM / NMFMA - i * NVMEM / NMFMA > 1) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    }
    if (i < NDS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);  // DS read
  }
}

// 16-byte-chunk XOR swizzle of an LDS row (CPR chunks).  A 16-byte fragment read serves 16 lanes
// = 16 consecutive rows per cycle; with 128-byte rows two rows share one 256-byte bank window, and
// (row parity, chunk ^ swz(row)) is distinct over the 16 rows, so the reads are conflict free.
// swz depends on r mod 16 only: the fragment addresses of a wavefront's 32-row MFMA blocks then
// differ by immediate offsets, and a copy's lane offset depends on its instruction only through
// the instruction's parity.
__device__ __forceinline__ int swz(int r) {
  if constexpr (CPR == 8) return (r >> 1) & 7;
  else return (r >> 1) & 3;
}

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding: vmcnt[3:0] in
// bits 3:0, vmcnt[5:4] in bits 15:14, expcnt 7 and lgkmcnt 15 = no wait).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}
__device__ __forceinline__ void wait_vmcnt_dyn(int n) {
  if (n >= 48) wait_vmcnt<48>();
  else if (n >= 32) wait_vmcnt<32>();
  else if (n >= 24) wait_vmcnt<24>();
  else if (n >= 16) wait_vmcnt<16>();
  else if (n >= 8) wait_vmcnt<8>();
  else if (n >= 4) wait_vmcnt<4>();
  else wait_vmcnt<0>();
}
// LDS/scalar counter to zero, vector memory unconstrained.
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// Workgroup barrier without a memory fence: the copies still in flight must stay in flight, so
// the waits are explicit (above); the empty asm statements keep the compiler from moving memory
// accesses across the barrier.
__device__ __forceinline__ void block_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

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

// XCD-aware tile mapping.  Workgroup ids are dispatched round-robin over the 8 XCDs, so the 256
// workgroups resident at a time are 256 consecutive ids.  Tiles are rastered in column groups of
// GROUP_M = 16 M-tiles, so 256 consecutive raster positions cover a 16 x 16 block of tiles; within
// each aligned run of 256 ids the ids are permuted so that XCD x computes the 4 x 8 sub-block
// (M-tiles 4 (x % 4) .. + 4, N-tiles 8 (x / 4) .. + 8) of that block: its 32 CUs then share 4 A
// and 8 B panels in the XCD's L2, and each panel is shared by 2 (A) or 4 (B) XCDs through the
// memory-side cache.  Returns false for workgroups beyond the tile grid.
__device__ __forceinline__ bool map_tile(int tm, int tn, int& tile_m, int& tile_n) {
  const int total = tm * tn;
  const int pid = blockIdx.x;
  if (pid >= total) return false;
  int idx = pid;
  if ((pid | 255) < total) {  // a complete run of 256 ids: XCD-blocked permutation
    const int xcd = pid & 7, slot = (pid >> 3) & 31;
    const int m = 4 * (xcd & 3) + (slot & 3), n = 8 * (xcd >> 2) + (slot >> 2);
    idx = (pid & ~255) + n * 16 + m;
  }
  const int group_sz = GROUP_M * tn;
  const int g = idx / group_sz;
  const int first_m = g * GROUP_M;
  const int gm = min(tm - first_m, GROUP_M);
  const int in = idx - g * group_sz;
  tile_m = first_m + in % gm;
  tile_n = in / gm;
  return true;
}

// DEEP_B: the B operand streams through three LDS stages (A through two; 5 x 32 KiB = all 160 KiB),
// so B is copied two slices ahead instead of one.  The main loop waits on copy latency (copies issued
// later in a slice measured 2-8 % slower), and the forward GEMM, whose tiles are short (K = d), runs
// 2.0-2.3 % faster this way; the dhidden and dW GEMMs ran 3-4 % and 0.5 % slower, so they keep two
// stages of each operand.
constexpr int LDS_DEEP_B = 5 * OPND_B;
static_assert(LDS_DEEP_B <= 163840 && LDS_DEEP_B >= LDS_B, "three-stage pipeline fits the LDS");

// Reference of the stored probabilities of chunk column n in a forward tile with maximum m: m itself,
// or with a.zr (token-reference layout) the column's reference logit r, clamped to m - kRefSpan where
// it lies further below (then, with mark, the chunk is flagged: its dz needs the explicit pass).
// Columns n >= N (padding) keep m.
__device__ __forceinline__ float tile_ref(const GemmArgs& a, float m, int n, int N, bool mark) {
  if (!a.zr || n >= N) return m;
  const float r = a.zr[n];
  if (r >= m - kRefSpan) return r;
  if (mark) *a.fb = 1;
  return m - kRefSpan;
}

template <typename T, int EPI, bool STORE_Q, bool KTAIL>
__global__ void __launch_bounds__(NT) k_gemm(GemmArgs a) {
  constexpr bool DEEP_B = EPI == EPI_FWD && sizeof(T) == 2;
  __shared__ __attribute__((aligned(16))) char smem[DEEP_B ? LDS_DEEP_B : LDS_B];

  int M = a.M, N = a.N, K = a.K;
  // rows of the chunk: every trained token for the forward, those with a surrogate gradient for the
  // gradient GEMMs
  int64_t rc = (int64_t)(EPI == EPI_FWD ? a.hdr->n_eff : a.hdr->n_grad) - a.c0;
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
  const int lane = tid & 63, wid = __builtin_amdgcn_readfirstlane(tid >> 6), wm = wid / WAVES_N, wn = wid % WAVES_N;
  const int lrow = lane & 31, lh = lane >> 5;

  // ---- operand panels as buffer resources: rows beyond M/N (and, with KTAIL, K chunks beyond K)
  // read as zero through the hardware range check; 32-bit offsets address one 256-row panel.
  const uint32_t lda_b = (uint32_t)(a.lda * (int64_t)sizeof(T)), ldb_b = (uint32_t)(a.ldb * (int64_t)sizeof(T));
  const int rows_a = min(kTile, M - tile_m * kTile), rows_b = min(kTile, N - tile_n * kTile);
  const __amdgpu_buffer_rsrc_t rsa = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(reinterpret_cast<const char*>(a.A) + (int64_t)tile_m * kTile * lda_b), (short)0,
      (int)((uint32_t)rows_a * lda_b), kBufferFlags);
  const __amdgpu_buffer_rsrc_t rsb = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(reinterpret_cast<const char*>(a.B) + (int64_t)tile_n * kTile * ldb_b), (short)0,
      (int)((uint32_t)rows_b * ldb_b), kBufferFlags);
  const int64_t Kb = (int64_t)K * sizeof(T);
  int nk = (int)((Kb + KS - 1) / KS);
  // split K: this workgroup covers slices [ks0, ks0 + nk) of the tile's K range
  int ks0 = 0;
  if (EPI != EPI_FWD && a.ksplit > 1) {
    ks0 = (int)blockIdx.y * a.kslices;
    nk = max(0, min(nk, ks0 + a.kslices) - ks0);
  }

  // Direct global->LDS copies (LDS DMA): one instruction moves 64 lanes x 16 bytes into 1 KiB of
  // LDS at consecutive addresses, i.e. RPI rows of one K slice.  Wave w fills rows
  // [w * IPW * RPI, (w + 1) * IPW * RPI) of each operand with IPW instructions; lane l of
  // instruction j carries row (w * IPW + j) * RPI + l / CPR into LDS slot l % CPR, which holds the
  // logical 16-byte K chunk (l % CPR) ^ swz(row).
  // The lane part of a copy's offset depends on the instruction only through its parity; the row
  // part is uniform and goes into the scalar offset.
  static_assert(RPI % 2 == 0 || RPI == 1, "copy geometry");
  uint32_t voa[2], vob[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int row = (wid * IPW + j) * RPI + lane / CPR;
    const int chunk = (lane % CPR) ^ swz(row);
    voa[j] = (uint32_t)(lane / CPR) * lda_b + chunk * 16;
    vob[j] = (uint32_t)(lane / CPR) * ldb_b + chunk * 16;
  }
  // Rows past the panel (ragged last tiles) read as zero because their vector offset alone is out of
  // range: 0x80000000 >= num_records (every 256-row panel is at most 2 GiB, checked by the host), so
  // the read stays inside the panel whether or not the hardware adds the scalar offset to the check.
  // A lane's row is r0 + lane / CPR; it is past the panel when r0 >= rows - lane / CPR.
  const int lim_a = rows_a - lane / CPR, lim_b = rows_b - lane / CPR;
  // copies of slice kt for the rows owned by wavefront w
  auto dma_w = [&](int kt, int w) {
    char* st = smem + (kt % NSTAGE) * STAGE_B;
    const uint32_t kb = (uint32_t)(kt + ks0) * KS;
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const uint32_t r0 = (uint32_t)((w * IPW + j) * RPI);
      uint32_t oa = (int)r0 < lim_a ? voa[j & 1] : 0x80000000u;
      uint32_t ob = (int)r0 < lim_b ? vob[j & 1] : 0x80000000u;
      if constexpr (KTAIL) {
        // chunks past the end of K would read the next row: push them out of range (zero fill)
        const int row = (w * IPW + j) * RPI + lane / CPR;
        const uint32_t ck = kb + (((lane % CPR) ^ swz(row)) * 16);
        if ((int64_t)ck >= Kb) {
          oa = 0x80000000u;
          ob = 0x80000000u;
        }
      }
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, LDSP(st + (w * IPW + j) * 1024), 16, oa, kb + r0 * lda_b, 0, 0);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, LDSP(st + OPND_B + (w * IPW + j) * 1024), 16, ob,
                                               kb + r0 * ldb_b, 0, 0);
    }
  };
  auto dma = [&](int kt) { dma_w(kt, wid); };
  // LDS offsets of slice kt's operand panels: two stages of A + B (STAGE_B each), or with DEEP_B
  // three B buffers at 0, 32, 64 KiB and two A buffers at 96, 128 KiB.
  auto off_a = [&](int kt) { return DEEP_B ? 3 * OPND_B + (kt % 2) * OPND_B : (kt % NSTAGE) * STAGE_B; };
  auto off_b = [&](int kt) { return DEEP_B ? (kt % 3) * OPND_B : (kt % NSTAGE) * STAGE_B + OPND_B; };
  // copies of one operand of slice kt (DEEP_B pipeline)
  auto dma_op = [&](bool op_a, int kt) {
    const uint32_t kb = (uint32_t)(kt + ks0) * KS;
#pragma unroll
    for (int j = 0; j < IPW; ++j) {
      const uint32_t r0 = (uint32_t)((wid * IPW + j) * RPI);
      uint32_t o = op_a ? ((int)r0 < lim_a ? voa[j & 1] : 0x80000000u) : ((int)r0 < lim_b ? vob[j & 1] : 0x80000000u);
      if constexpr (KTAIL) {
        const int row = (wid * IPW + j) * RPI + lane / CPR;
        const uint32_t ck = kb + (((lane % CPR) ^ swz(row)) * 16);
        if ((int64_t)ck >= Kb) o = 0x80000000u;
      }
      if (op_a)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsa, LDSP(smem + off_a(kt) + (wid * IPW + j) * 1024), 16, o,
                                                 kb + r0 * lda_b, 0, 0);
      else
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsb, LDSP(smem + off_b(kt) + (wid * IPW + j) * 1024), 16, o,
                                                 kb + r0 * ldb_b, 0, 0);
    }
  };
  // Fragment reads: lane (lrow, lh) takes logical K chunk 2 kk + lh of row r.
  auto frags = [&](int kt, int kk, u32x4 (&fa)[MBW], u32x4 (&fb)[NBW]) {
    const char* sA = smem + off_a(kt);
    const char* sB = smem + off_b(kt);
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb) {
      const int r = wm * WTM + mb * 32 + lrow;
      fa[mb] = *reinterpret_cast<const u32x4*>(sA + r * KS + (((2 * kk + lh) ^ swz(r)) * 16));
    }
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
      const int r = wn * WTN + nb * 32 + lrow;
      fb[nb] = *reinterpret_cast<const u32x4*>(sB + r * KS + (((2 * kk + lh) ^ swz(r)) * 16));
    }
  };

  f32x16 acc[MBW][NBW];
#pragma unroll
  for (int i = 0; i < MBW; ++i)
#pragma unroll
    for (int j = 0; j < NBW; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;
  auto mma = [&](const u32x4 (&fa)[MBW], const u32x4 (&fb)[NBW]) {
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
      for (int nb = 0; nb < NBW; ++nb) Op<T>::mma(acc[mb][nb], fa[mb], fb[nb]);
  };

  // Pipeline over K slices with NSTAGE LDS buffers: the copy of slice kt + NSTAGE is issued
  // right after the barrier that retires slice kt, so every copy has NSTAGE - 1 slices of MFMA
  // work to land.  Within a slice, the fragments of K step kk + 1 are read under the MFMAs of
  // step kk; at the last step this wave's copies of slice kt + 1 are awaited, one barrier
  // publishes every wave's copies (and retires slice kt), slice kt + NSTAGE is issued into the
  // freed buffer and the first fragments of slice kt + 1 are read.
  u32x4 f0a[MBW], f0b[NBW], f1a[MBW], f1b[NBW];
  if constexpr (DEEP_B) {
    // Three-stage B: at the end of slice kt the A copies of slice kt + 2 and then the B copies of slice
    // kt + 3 are issued, so when slice kt + 1 is awaited only the newest B batch may still be in flight.
    if (nk > 0) {
      dma_op(true, 0);
      dma_op(false, 0);
    }
    if (nk > 1) {
      dma_op(true, 1);
      dma_op(false, 1);
    }
    if (nk > 2) dma_op(false, 2);
    if (nk > 0) {
      if (nk > 2) wait_vmcnt<3 * IPW>();
      else wait_vmcnt<0>();
      block_barrier();
      frags(0, 0, f0a, f0b);
    }
  } else {
    const int npro = min(nk, NSTAGE);
    for (int s = 0; s < npro; ++s) dma(s);
    if (nk > 0) {
      wait_vmcnt_dyn(DMA_PER_SLICE * (npro - 1));
      block_barrier();
      frags(0, 0, f0a, f0b);
    }
  }
  // steady state: every copy the loop issues lies inside [0, nk)
  const int ahead = DEEP_B ? 3 : NSTAGE;
  int kt = 0;
  for (; kt + ahead < nk; ++kt) {
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      u32x4(&ca)[MBW] = (kk & 1) ? f1a : f0a;
      u32x4(&cb)[NBW] = (kk & 1) ? f1b : f0b;
      u32x4(&na)[MBW] = (kk & 1) ? f0a : f1a;
      u32x4(&nb)[NBW] = (kk & 1) ? f0b : f1b;
      if (kk + 1 < NKK) {
        frags(kt, kk + 1, na, nb);
        mma(ca, cb);
        sched_step<MBW * NBW, MBW + NBW, 0>();
      } else {
        if constexpr (DEEP_B) wait_vmcnt<IPW>();  // slice kt+1 has landed; B of slice kt+2 may be in flight
        else wait_vmcnt<DMA_PER_SLICE * (NSTAGE - 2)>();  // slice kt+1 has landed
        wait_lgkm0();
        block_barrier();
        if constexpr (DEEP_B) {
          dma_op(true, kt + 2);
          dma_op(false, kt + 3);
        } else {
          dma(kt + NSTAGE);
        }
        frags(kt + 1, 0, na, nb);
        mma(ca, cb);
        sched_step<MBW * NBW, MBW + NBW, DMA_PER_SLICE>();
      }
    }
  }
  for (; kt < nk; ++kt) {
    // drain: the last copies (DEEP_B: the A copies of the last slice), no interleaving
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) {
      u32x4(&ca)[MBW] = (kk & 1) ? f1a : f0a;
      u32x4(&cb)[NBW] = (kk & 1) ? f1b : f0b;
      u32x4(&na)[MBW] = (kk & 1) ? f0a : f1a;
      u32x4(&nb)[NBW] = (kk & 1) ? f0b : f1b;
      if (kk + 1 < NKK) {
        frags(kt, kk + 1, na, nb);
      } else if (kt + 1 < nk) {
        if constexpr (DEEP_B) wait_vmcnt<0>();
        else wait_vmcnt_dyn(DMA_PER_SLICE * min(nk - 2 - kt, NSTAGE - 2));
        wait_lgkm0();
        block_barrier();
        if constexpr (DEEP_B) {
          if (kt + 2 < nk) dma_op(true, kt + 2);
        }
        frags(kt + 1, 0, na, nb);
      }
      mma(ca, cb);
    }
  }
  // the epilogues reuse the LDS of the pipeline
  wait_lgkm0();
  block_barrier();

  // ------------------------------------------------------------------ epilogues
  // Accumulator (mb, nb, r) of this lane sits at tile row wm*WTM + mb*32 + 8*(r/4) + 4*lh + r%4 and
  // tile column wn*WTN + nb*32 + lrow.
  if constexpr (EPI != EPI_FWD) {
    if (a.ksplit > 1) {
      // split K: fp32 partial of this K range; the reduction kernel applies the epilogue
      float* part = a.part + (int64_t)blockIdx.y * a.mp * a.ldp;
#pragma unroll
      for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rl = tile_m * kTile + wm * WTM + mb * 32 + (r >> 2) * 8 + lh * 4 + (r & 3);
          if (rl < M) {
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) {
              const int cl = tile_n * kTile + wn * WTN + nb * 32 + lrow;
              if (cl < N) part[(int64_t)rl * a.ldp + cl] = acc[mb][nb][r];
            }
          }
        }
      return;
    }
  }
  if constexpr (EPI == EPI_FWD) {
    // rows = vocabulary v = v0 + rl, columns = chunk-local token n.  Logits z = (W h) / tau.
    if (a.inv_tau != 1.0f) {
#pragma unroll
      for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) acc[mb][nb] *= a.inv_tau;
    }
    const int v0 = tile_m * kTile;
    const int V = a.V;
    const bool full_v = v0 + kTile <= V;
    // q and q^T are read only for the tokens with a surrogate gradient (the first n_grad of the
    // list): the stores stop there (q^T writes zero columns up to the K pad)
    int ng = N;
    if constexpr (STORE_Q) {
      const int64_t g = (int64_t)a.hdr->n_grad - a.c0;
      ng = g < 0 ? 0 : (g < N ? (int)g : N);
    }
    float* red_m = reinterpret_cast<float*>(smem + RED_OFF);  // [WAVES_M][256]
    float* red_s = red_m + WAVES_M * kTile;                    // [WAVES_M][256]
    float* red_u = red_s + WAVES_M * kTile;                    // [WAVES_M][256]

    // phase 1: per-token max over this tile's 256 vocabulary rows; gather the target logit.
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
      const int cl = wn * WTN + nb * 32 + lrow;
      const int n = tile_n * kTile + cl;
      float mx = -INFINITY;
#pragma unroll
      for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int rl = wm * WTM + mb * 32 + (r >> 2) * 8 + lh * 4 + (r & 3);
          const float z = (full_v || v0 + rl < V) ? acc[mb][nb][r] : -INFINITY;
          mx = fmaxf(mx, z);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      if (lh == 0) red_m[wm * kTile + cl] = mx;
      if (n < N) {
        const int y = a.ytgt[a.c0 + n];
        const int yl = y - v0 - wm * WTM;
        if (y >= 0 && y < V && yl >= 0 && yl < WTM && ((yl >> 2) & 1) == lh) {
          const int tmb = yl >> 5, tr = ((yl & 31) >> 3) * 4 + (yl & 3);
          float z = 0.0f;
#pragma unroll
          for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
            for (int r = 0; r < 16; ++r) z = (mb == tmb && r == tr) ? acc[mb][nb][r] : z;
          a.zy[a.c0 + n] = z;
        }
      }
    }
    __syncthreads();

    // phase 2: e = exp(z - c), s = sum e, u = sum e (z - c) against the token's reference c (the
    // tile maximum m, or with a.zr the reference logit r clamped to m - kRefSpan); e optionally
    // staged for storage.
    char* sQ = smem;
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
      const int cl = wn * WTN + nb * 32 + lrow;
      float mt = red_m[cl];
#pragma unroll
      for (int w = 1; w < WAVES_M; ++w) mt = fmaxf(mt, red_m[w * kTile + cl]);
      const float ref = tile_ref(a, mt, tile_n * kTile + cl, N, true);
      const float mt2 = ref * kLog2e;
      float s = 0.0f, u = 0.0f;
#pragma unroll
      for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          float ev[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int r = g * 4 + i;
            const int rl = wm * WTM + mb * 32 + g * 8 + lh * 4 + i;
            const float z = acc[mb][nb][r];
            const bool valid = full_v || v0 + rl < V;
            const float e = valid ? __builtin_amdgcn_exp2f(fmaf(z, kLog2e, -mt2)) : 0.0f;
            s += e;
            u = fmaf(e, z - ref, u);
            ev[i] = e;
          }
          if constexpr (STORE_Q) {
            const int rl0 = wm * WTM + mb * 32 + g * 8 + lh * 4;
            if constexpr (sizeof(T) == 2) {
              u32x2 pk;
              pk.x = pack_bf16x2(ev[0], ev[1]);
              pk.y = pack_bf16x2(ev[2], ev[3]);
              *reinterpret_cast<u32x2*>(sQ + cl * QROW + (((rl0 >> 3) ^ qswz(cl)) << 4) + (rl0 & 7) * 2) = pk;
            } else {
              const int n = tile_n * kTile + cl;
              if (n < ng) {
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
      for (int nb = 0; nb < NBW; ++nb) {
        const int cl = wn * WTN + nb * 32 + lrow;
        const int n = tile_n * kTile + cl;
        if (n < N) {
          float m = red_m[cl], s = red_s[cl], u = red_u[cl];
#pragma unroll
          for (int w = 1; w < WAVES_M; ++w) {
            m = fmaxf(m, red_m[w * kTile + cl]);
            s += red_s[w * kTile + cl];
            u += red_u[w * kTile + cl];
          }
          const int64_t o = (int64_t)tile_m * a.Mc + n;
          a.pm[o] = tile_ref(a, m, n, N, false);
          a.ps[o] = s;
          a.pu[o] = u;
        }
      }
    }
    if constexpr (STORE_Q && sizeof(T) == 2) {
      // phase 3: coalesced copy of the staged bf16 tile to q[n][v0 .. v0 + 255].  q is read once,
      // by the dz kernel or the dhidden GEMM after this launch: non-temporal stores keep it from
      // displacing the operand panels that later tiles of this launch re-read from the caches.
      const int chunk = tid & 31;
#pragma unroll 4
      for (int it = 0; it < kTile * 32 / NT; ++it) {
        const int cl = (tid >> 5) + (NT / 32) * it;
        const int n = tile_n * kTile + cl;
        if (n < ng) {
          const u32x4 v = *reinterpret_cast<const u32x4*>(sQ + cl * QROW + ((chunk ^ qswz(cl)) << 4));
          char* dst = reinterpret_cast<char*>(a.q) + ((int64_t)n * a.ldq + v0) * 2 + chunk * 16;
          __builtin_nontemporal_store(v, reinterpret_cast<u32x4*>(dst));
        }
      }
      if (a.qt) {
        // phase 4: the same tile transposed into q^T[v0 .. v0 + 255][tokens of the tile], the dW
        // GEMM's operand (columns of tokens >= n_grad as zero, up to the K pad).  Each lane transposes
        // an 8 x 8 square in registers: wavefront w covers the 16 x 256 blocks (vocabulary rows x
        // tokens) w and w + 8, lane (a8, b8) = (lane / 32, lane % 32) the vocabulary rows 8 a8 .. + 7
        // and tokens 8 b8 .. + 7 of a block, so each store writes two rows of 512 contiguous bytes
        // (8 rows of 128 bytes per store measured 1.5 ms per step slower).  With the chunk swizzle the
        // reads of 8 consecutive lanes fall in distinct bank groups.
        const int a8 = lane >> 5, b8 = lane & 31;
        const int ngpad = (ng + kKAlign - 1) / kKAlign * kKAlign;
#pragma unroll
        for (int it = 0; it < kTile * kTile / 4096 / NWAVE; ++it) {
          const int blk = wid + NWAVE * it;
          const int rl0 = blk * 16 + a8 * 8, cl0 = b8 * 8;
          const int n0 = tile_n * kTile + cl0;
          if (n0 >= ngpad) continue;
          u32x4 in[8];
#pragma unroll
          for (int j = 0; j < 8; ++j)
            in[j] = n0 + j < ng
                        ? *reinterpret_cast<const u32x4*>(sQ + (cl0 + j) * QROW + (((rl0 >> 3) ^ qswz(cl0 + j)) << 4))
                        : u32x4{0, 0, 0, 0};
#pragma unroll
          for (int k = 0; k < 8; ++k) {
            u32x4 o;
#pragma unroll
            for (int m = 0; m < 4; ++m) {
              const uint32_t lo = in[2 * m][k >> 1], hi = in[2 * m + 1][k >> 1];
              o[m] = (k & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
            }
            char* dst = reinterpret_cast<char*>(a.qt) + ((int64_t)(v0 + rl0 + k) * a.ldqt + n0) * 2;
            __builtin_nontemporal_store(o, reinterpret_cast<u32x4*>(dst));
          }
        }
      }
    }
  } else if constexpr (EPI == EPI_DH) {
    // rows = chunk-local tokens, columns = hidden features; scatter to dh[idx[c0 + row]].
    // With row scales (token-reference layout), dh = diag(s) (q W^T).
    T* out = reinterpret_cast<T*>(a.out);
    const bool scaled = a.rs != nullptr && *a.rs_off == 0;
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = tile_m * kTile + wm * WTM + mb * 32 + (r >> 2) * 8 + lh * 4 + (r & 3);
        if (rl < M) {
          const int64_t row = a.idx[a.c0 + rl];
          const float sc = scaled ? a.rs[rl] : 1.0f;
#pragma unroll
          for (int nb = 0; nb < NBW; ++nb) {
            const int cl = tile_n * kTile + wn * WTN + nb * 32 + lrow;
            if (cl < N) store_elem<T>(out + row * a.ldo + cl, acc[mb][nb][r] * sc);
          }
        }
      }
  } else {
    // rows = vocabulary, columns = hidden features; fp32 dW, overwritten by the first
    // chunk unless the caller accumulates.
    const bool add = a.accumulate || a.c0 > 0;
#pragma unroll
    for (int mb = 0; mb < MBW; ++mb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int rl = tile_m * kTile + wm * WTM + mb * 32 + (r >> 2) * 8 + lh * 4 + (r & 3);
        if (rl < M) {
#pragma unroll
          for (int nb = 0; nb < NBW; ++nb) {
            const int cl = tile_n * kTile + wn * WTN + nb * 32 + lrow;
            if (cl < N) {
              float* p = a.dw + (int64_t)rl * a.ldo + cl;
              *p = add ? *p + acc[mb][nb][r] : acc[mb][nb][r];
            }
          }
        }
      }
  }
}

// Split-K reduction: out = sum of the partials in split order (deterministic), then the dhidden
// scatter or the dW overwrite / accumulate.  Rows and the empty-chunk rule follow the GEMM.
template <typename T, int EPI>
__global__ void __launch_bounds__(256) k_splitk_reduce(GemmArgs a) {
  int64_t rc = (int64_t)a.hdr->n_grad - a.c0;
  rc = rc < 0 ? 0 : (rc > a.Mc ? a.Mc : rc);
  int M = a.M;
  if (EPI == EPI_DH) M = (int)rc;
  if (EPI == EPI_DW && rc == 0 && a.c0 > 0) return;
  const int N = a.N;
  const int64_t total = (int64_t)M * N;
  const bool add = EPI == EPI_DW && (a.accumulate || a.c0 > 0);
  for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total; e += (int64_t)gridDim.x * blockDim.x) {
    const int64_t m = e / N, n = e - m * N;
    float acc = 0.0f;
    for (int y = 0; y < a.ksplit; ++y) acc += a.part[((int64_t)y * a.mp + m) * a.ldp + n];
    if constexpr (EPI == EPI_DH) {
      const int64_t row = a.idx[a.c0 + m];
      if (a.rs && *a.rs_off == 0) acc *= a.rs[m];
      store_elem<T>(reinterpret_cast<T*>(a.out) + row * a.ldo + n, acc);
    } else {
      float* p = a.dw + m * a.ldo + n;
      *p = add ? *p + acc : acc;
    }
  }
}

inline unsigned tiles(int64_t n) { return (unsigned)((n + kTile - 1) / kTile); }

template <typename T, int EPI>
hipError_t grad_impl(const GemmArgs& a, unsigned ntiles, hipStream_t s) {
  const unsigned ny = a.ksplit > 1 ? (unsigned)a.ksplit : 1u;
  k_gemm<T, EPI, false, false><<<dim3(ntiles, ny), NT, 0, s>>>(a);
  if (a.ksplit > 1) {
    const int64_t total = (int64_t)a.M * a.N;
    const unsigned blocks = (unsigned)std::min<int64_t>((total + 255) / 256, 8192);
    k_splitk_reduce<T, EPI><<<blocks, 256, 0, s>>>(a);
  }
  return hipGetLastError();
}

template <typename T>
hipError_t fwd_impl(const GemmArgs& a, bool store_q, hipStream_t s) {
  dim3 grid(tiles(a.M) * tiles(a.Mc));
  const bool ktail = ((int64_t)a.K * (int64_t)sizeof(T)) % KS != 0;
  if (store_q) {
    if (ktail) k_gemm<T, EPI_FWD, true, true><<<grid, NT, 0, s>>>(a);
    else k_gemm<T, EPI_FWD, true, false><<<grid, NT, 0, s>>>(a);
  } else {
    if (ktail) k_gemm<T, EPI_FWD, false, true><<<grid, NT, 0, s>>>(a);
    else k_gemm<T, EPI_FWD, false, false><<<grid, NT, 0, s>>>(a);
  }
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
  const unsigned nt = tiles(a.Mc) * tiles(a.N);
  prof_mark(KK_DH_GEMM, true, s);
  hipError_t e = dtype == RLK_DTYPE_BF16 ? grad_impl<bf16_t, EPI_DH>(a, nt, s) : grad_impl<float, EPI_DH>(a, nt, s);
  prof_mark(KK_DH_GEMM, false, s);
  return e;
}

hipError_t launch_dw_gemm(int dtype, const GemmArgs& a, hipStream_t s) {
  const unsigned nt = tiles(a.M) * tiles(a.N);
  prof_mark(KK_DW_GEMM, true, s);
  hipError_t e = dtype == RLK_DTYPE_BF16 ? grad_impl<bf16_t, EPI_DW>(a, nt, s) : grad_impl<float, EPI_DW>(a, nt, s);
  prof_mark(KK_DW_GEMM, false, s);
  return e;
}

}  // namespace rlk
