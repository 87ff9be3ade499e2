// Fused attention forward for gfx950 (MI355X) with the softmax exponential
// either the hardware exp2 (control) or Rowmax-H15 (Sec. 5.2 Eq. (m-h15),
// App. B.1 "Implementation") and its finer input roundings S(Q_{2^-k})
// (App. B.2), or Rowmax-PoT (App. A.6), behind the C ABI declared in
// h15attn.h.
//
// Kernel structure (one workgroup = 4 wave64s for FP8, 8 or 4 for BF16; 32 query
// rows of one head per wave; two waves per SIMD, three for FP8 at d = 64):
//   * each wave keeps its 32 query rows of Q in VGPRs as the MFMA B operand,
//     brought in through LDS with whole-row loads;
//   * key tiles of 128 keys are copied HBM -> LDS with buffer loads that
//     write LDS directly (no staging registers), double-buffered (the copy
//     of tile t+1 is in flight while tile t is computed, one barrier per
//     tile) or single-buffered (K(t+1) copied while the weights and PV of
//     tile t run, V(t+1) while QK^T of tile t+1 runs, two barriers per tile:
//     the lattice weights at FP8 d = 128, and the compact BF16 layout);
//   * scores are computed transposed, S^T = K Q^T, with 32x32 MFMAs (bf16
//     32x32x16, fp8 32x32x64): each lane owns one query row and 64 of the
//     tile's 128 keys, so the row max and row sum are in-lane reductions plus
//     one exchange with lane ^ 32;
//   * the weights are produced in VALU registers (hardware exp2, or the
//     lattice weights finished two at a time in 16-bit lanes), converted to
//     the MFMA operand type and used directly as the B operand of
//     O^T += V^T P^T: the MFMA contraction index is mapped to keys so that
//     the S accumulator layout already is the P operand layout;
//   * V is read from LDS with the transposing reads ds_read_b64_tr_b16 (bf16)
//     and ds_read_b64_tr_b8 (fp8), in the matching key order;
//   * at fp8 the PV MFMAs over the tile's first 64 keys go first, and the
//     weights of the other 64 are finished between them (split P), so that
//     a wave's VALU work overlaps its own matrix-core work;
//   * O leaves through LDS, so that each store covers whole rows.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <mutex>
#include <type_traits>

#include "attn_params.h"
#include "h15attn.h"

// The file is compiled twice (build.py): with H15_FP8_LATTICE_D128 = 1 it
// holds only the forward kernels of the FP8 lattice weights at d = 128 and
// their launcher, built with the iterative ILP machine scheduler (measured at
// FP8 8K: +1.2% causal, +1.4% non-causal; the exact control and the BF16 and
// d = 64 kernels are better off with the default scheduler, which at d = 64
// keeps three waves per SIMD); with 0, the default, everything else.
#ifndef H15_FP8_LATTICE_D128
#define H15_FP8_LATTICE_D128 0
#endif

namespace h15 {
hipError_t launch_fwd_fp8_lattice128(const Params& p, bool causal, int mode, hipStream_t st, bool probe);
}

namespace {

using namespace h15;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x2v __attribute__((__vector_size__(2 * sizeof(int))));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x2 __attribute__((ext_vector_type(2)));

#define LDS_PTR(T, p) ((__attribute__((address_space(3))) T*)(p))

enum { DT_BF16 = 0, DT_FP8 = 1 };

// Waves per workgroup in the default layout: 4 for FP8 (two workgroups
// share a CU, so one's barrier and prologue stalls overlap the other's
// work), 8 for BF16 (whose double-buffered tiles at d = 128 leave LDS for
// only one workgroup per CU; the compact layout, Cfg below, has 4).
template <int DT>
constexpr int waves_per_group() {
  return DT == DT_FP8 ? 4 : 8;
}
constexpr int MAX_THREADS = 8 * 64;
// LDS operand prefetch distance (in MFMAs) of the QK^T and PV products
constexpr int QK_AHEAD = 3;
constexpr int PV_AHEAD = 3;
// word 3 of a raw buffer resource on CDNA (32-bit data format, no swizzle)
constexpr int BUF_DWORD3 = 0x00020000;
// instruction classes of __builtin_amdgcn_sched_group_barrier
constexpr int SG_MFMA = 0x008;
constexpr int SG_DS_READ = 0x100;
constexpr float H15_MAGIC = 12582912.0f;  // 0x4B400000 = 2^23 + 2^22
// top half of bits(1.0) in both 16-bit lanes
constexpr uint32_t ONE_BITS16X2 = 0x3F803F80u;

// Kernel weight modes (attn_params.h): the order k of a lattice mode, and its
// clamp form.
constexpr int mode_order(int mode) { return (mode + 1) / 2; }
constexpr bool mode_lattice(int mode) { return mode != MODE_EXACT && mode != MODE_ROWMAX_POT; }
constexpr bool mode_narrow(int mode) { return mode_lattice(mode) && mode % 2 == 0; }
constexpr int POT_KMAX = 20;  // tail clamp of Rowmax-PoT

// CMP: the compact layout for grids that underfill the chip (BF16, chosen
// per call on the host): 4 waves per group and at most 80 KB of LDS, so two
// groups share a CU and one's prologue, barriers and epilogue overlap the
// other's work; at d = 128 that means single-buffered K and V tiles.
template <int DT, int D, bool CMP = false>
struct Cfg {
  static constexpr int EB = DT == DT_BF16 ? 2 : 1;  // operand bytes
  static constexpr int RB = D * EB;                 // bytes per K/V row
  static constexpr int NCH = RB / 16;               // 16-byte chunks per row
  static constexpr int TILE = BC * RB;              // bytes of one K (or V) tile
  static constexpr int BUF = 2 * TILE;              // K then V
  static constexpr int CHUNKS = BC * NCH;           // 16-byte chunks per tile
  static constexpr int NW = CMP ? 4 : waves_per_group<DT>();  // waves per workgroup
  static constexpr int BR = NW * WROWS;                       // query rows per workgroup
  // K/V tile buffers: two (the copy of tile t + 1 overlaps tile t), or one
  // when two would not let two compact groups share a CU's 160 KB of LDS
  static constexpr int NSTAGE = (CMP && 2 * BUF > 80 * 1024) ? 1 : 2;
  static_assert(CHUNKS % (NW * 64) == 0, "tile/staging mismatch");
  static_assert(BR == (CMP ? FWD_ROWS_COMPACT : DT == DT_FP8 ? FWD_ROWS_FP8 : FWD_ROWS_BF16),
                "row block of attn_params.h");
};

// Bank-spreading XOR swizzles of the 16-byte chunks of a row.  K rows are read
// as the MFMA A operand (one chunk of 32 consecutive rows per instruction);
// V rows through the transposing reads (4 rows x 2 chunks for bf16, 8 rows x
// 1 chunk for fp8 per 16 lanes).  An fp8 row is 128 bytes, half the banks'
// width, so rows r and r + 1 start on different bank halves; the K swizzle
// then varies with r / 2, so that 16 consecutive rows reading one logical
// chunk cover every bank once (with r % NCH, rows r and r + 8 shared banks;
// the counter read 2,080 conflict cycles per wave at d = 128, now zero).
template <int DT, int D>
__device__ __forceinline__ int k_swz(int row) {
  using C = Cfg<DT, D>;
  if constexpr (DT == DT_BF16) return row % C::NCH;
  else return (row >> 1) % C::NCH;
}
template <int DT, int D>
__device__ __forceinline__ int v_swz(int row) {
  using C = Cfg<DT, D>;
  if constexpr (DT == DT_BF16) return ((C::NCH >= 16 ? 4 : 2) * (row & 3)) % C::NCH;
  else return ((row & 3) | (((row >> 3) & 1) << 2)) % C::NCH;
}

__device__ __forceinline__ void map_block(const Params& p, int L, int& qb, int& b, int& h) {
  const int nbh = p.B * p.Hq;
  if (p.remap) {
    // Hardware workgroup ids go round-robin over the 8 XCDs (id mod 8).  Give
    // each XCD whole key/value-head groups, so the query heads that read the
    // same K/V share one L2, and walk query blocks longest-first.
    const int x = L & 7, j = L >> 3;
    int qi, kvl, gi;
    if (p.remap == 2) {
      // one KV head group at a time per XCD: the K/V working set of the
      // workgroups resident on an XCD is one head's (non-causal, where every
      // query block reads all of it)
      const int span = p.nqb * p.G;
      kvl = j / span;
      const int r = j - kvl * span;
      qi = r / p.G;
      gi = r - qi * p.G;
    } else {
      const int per = nbh >> 3;
      qi = j / per;
      const int loc = j - qi * per;
      kvl = loc / p.G;
      gi = loc - kvl * p.G;
    }
    qb = p.nqb - 1 - qi;
    const int kvg = kvl * 8 + x;
    b = kvg / p.Hkv;
    h = (kvg - b * p.Hkv) * p.G + gi;
  } else {
    const int qi = L / nbh, bh = L - qi * nbh;
    qb = p.nqb - 1 - qi;
    b = bh / p.Hq;
    h = bh - b * p.Hq;
  }
}

// Weight of one score, S(Q_{2^-k}(x)) with k = mode_order(MODE) (App. B.1
// "Implementation" for k = 1, App. B.2 "Exponential-map ablation" for k = 2,
// 3): y = 2^k x = fma(s, 2^k c1, nb), clamp at -126 * 2^k, RNE add of
// 0x4B400000 (n = RNE(y) lands in the low mantissa bits), left shift by
// 23 - k (the low k bits of n become the top mantissa bits, the rest the
// exponent), plus the bits of 1.0, all modulo 2^32.
//
// Such a weight has at most k <= 3 mantissa bits, so the low 16 bits of its
// FP32 pattern are zero and its top 16 bits, (n << (7 - k)) + 0x3F80 modulo
// 2^16, are its exact BF16 pattern.  The kernel finishes the weights two at
// a time in the 16-bit lanes of one register: the row sum takes one
// two-element dot product per pair, and the pair is already a BF16 operand
// (or one packed conversion away from FP8).
//
// sq_pre: the 32-bit value whose low half carries n: bits(max(y, -126 2^k) +
// magic), or for the narrow clamp bits(y + magic) (the magic's low half is
// zero, so the low half is n modulo 2^16).
template <int MODE>
__device__ __forceinline__ uint32_t sq_pre(float s, float ck, float nbk) {
  constexpr int K = mode_order(MODE);
  const float y = __builtin_fmaf(s, ck, nbk);
  if constexpr (mode_narrow(MODE)) return __float_as_uint(y + H15_MAGIC);
  else return __float_as_uint(__builtin_fmaxf(y, -126.0f * (float)(1 << K)) + H15_MAGIC);
}

// The BF16 weights of two keys in one word (u0 in the low lane): the low
// halves of their sq_pre values, the narrow clamp max(n, -126 2^k) on int16
// lanes (n is then n itself: the launcher selects the narrow mode only when
// every |y| is provably below 2^15), and n 2^(7-k) + 0x3F80 per lane modulo
// 2^16 in one packed multiply-add.
template <int MODE>
__device__ __forceinline__ uint32_t sq_pack(uint32_t u0, uint32_t u1) {
  constexpr int K = mode_order(MODE);
  uint32_t x = __builtin_amdgcn_perm(u1, u0, 0x05040100u);
  if constexpr (mode_narrow(MODE)) {
    constexpr short lo = (short)(-126 * (1 << K));
    x = __builtin_bit_cast(uint32_t, __builtin_elementwise_max(__builtin_bit_cast(i16x2, x), i16x2{lo, lo}));
  }
  // the multiplier is an inline constant read from its low half in both
  // lanes (op_sel_hi 0); the addend comes from a scalar register
  uint32_t r;
  asm("v_pk_mad_u16 %0, %1, %2, %3 op_sel_hi:[1,0,1]" : "=v"(r) : "v"(x), "n"(1 << (7 - K)), "s"(ONE_BITS16X2));
  return r;
}

// sq_pre value of a masked key: its packed weight is +0.  n = 385 * 2^k gives
// n 2^(7-k) = 0xC080 = -0x3F80 modulo 2^16, and lies above the narrow clamp.
template <int MODE>
constexpr uint32_t sq_masked() {
  return 385u << mode_order(MODE);
}
// (0x4B3F0000 | sq_masked) = 0x1.8p23 - 2^16 + sq_masked lies below
// 0x1.8p23 - 2^15 for every mode
static_assert((385u << 3) < (1u << 15), "the lift stays below every narrow-mode t");

// init plus the row sum of a tile's packed weights: one dot product with
// (1, 1) per word, in two chains.
__device__ __forceinline__ float dot2_ones(uint32_t w, float acc) {
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), ones, acc, false);
}

__device__ __forceinline__ float pair_sum(const uint32_t (&w)[4][8], float init) {
  const bf16x2 ones = {(__bf16)1.0f, (__bf16)1.0f};
  float a[2] = {init, 0.0f};
#pragma unroll
  for (int kb = 0; kb < 4; ++kb)
#pragma unroll
    for (int q = 0; q < 8; ++q)
      a[q & 1] = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w[kb][q]), ones, a[q & 1], false);
  return a[0] + a[1];
}

// Rowmax-PoT weight of one score (App. A.6 Eq. (rowmax-pot)) against the
// whole-row maximum m: base-two gap x = fp32(fp32(m - s) c1), d = min(K_max,
// floor(x + 1/2)) (exact: x + 1/2 is representable below 2^22), w = 2^-d.
__device__ __forceinline__ float pot_weight(float s, float m, float c1) {
  const float x = (m - s) * c1;
  const float d = __builtin_fminf(__builtin_floorf(x + 0.5f), (float)POT_KMAX);
  return __builtin_amdgcn_ldexpf(1.0f, -(int)d);
}

// x, or y where key offset C lies beyond this lane's last valid offset lim.
// Compare and select go through VCC together (C as an immediate): written
// as plain C the compiler keeps all 64 masks of a tile live in scalar
// registers at once.
template <int C>
__device__ __forceinline__ float select_beyond(int lim, float x, float y) {
  float r;
  // volatile: keeps the masking inside the branch that needs it
  asm volatile("v_cmp_gt_i32 vcc, %1, %2\n\tv_cndmask_b32 %0, %3, %4, vcc"
               : "=v"(r)
               : "n"(C), "v"(lim), "v"(x), "v"(y)
               : "vcc");
  return r;
}
// y over the scores of a tile whose key offset lies beyond lim
template <int E = 0>
__device__ __forceinline__ void mask_beyond(f32x16 (&v)[4], int lim, float y) {
  if constexpr (E < 64) {
    constexpr int kb = E / 16, j = E % 16;
    v[kb][j] = select_beyond<kb * 32 + 8 * (j >> 2) + (j & 3)>(lim, v[kb][j], y);
    mask_beyond<E + 1>(v, lim, y);
  }
}

// This lane's value and that of lane i ^ 32 (in an order that depends on the
// lane), exchanged on the VALU rather than through LDS.
__device__ __forceinline__ void with_partner(float x, float& a, float& b) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  a = __uint_as_float(r[0]);
  b = __uint_as_float(r[1]);
}

// Compile-time loop: f(integral_constant<int, I>) for I in [B, E).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// Transposing LDS reads written as inline asm.  The compiler's wait counting
// would make the intrinsic forms wait for every LDS copy in flight (it cannot
// tell that those copies land in other buffers); here the caller waits for
// the reads itself with lds_wait, which also orders the uses after the wait.
template <int OFF>
__device__ __forceinline__ i32x2v ds_read_tr8(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset");
  i32x2v r;
  asm volatile("ds_read_b64_tr_b8 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "n"(OFF));
  return r;
}
template <int OFF>
__device__ __forceinline__ i32x2v ds_read_tr16(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "ds offset");
  i32x2v r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "n"(OFF));
  return r;
}
// Wait until at most N LDS operations of this wave are outstanding (they
// complete in order), then hand x on as produced after the wait.
template <int N, typename T>
__device__ __forceinline__ void lds_wait(T& x) {
  static_assert(N >= 0 && N < 16, "lgkmcnt range");
  asm volatile("s_waitcnt lgkmcnt(%1)" : "+v"(x) : "n"(N));
}

// The scores of a tile are next read by inline asm (the v_max3_f32 tree of
// tile_max, and the compare/select of the masking), and the compiler inserts
// no wait states between a matrix-core write and an inline-asm read.  This
// statement does: it takes the four score blocks as in/out operands, so it
// comes after the last QK^T MFMA and every later read of the blocks comes
// after it, and it holds the wave for 24 wait states, more than the 20 that
// gfx950 requires between a 16-pass XDL write of a VGPR and a VALU read of
// it (the shorter MFMAs need fewer).  (Reading a block right after its MFMA,
// with no such wait, was measured to return stale values.)
__device__ __forceinline__ void settle_scores(f32x16 (&v)[4]) {
  asm("s_nop 15\n\ts_nop 7" : "+v"(v[0]), "+v"(v[1]), "+v"(v[2]), "+v"(v[3]));
}

// Tree reductions over a lane's 64 scores (short dependency chains).  The
// maximum is taken with v_max3_f32 directly: fmaxf on matrix-core results
// would first canonicalize every input (one extra instruction per score).
// Its reads of the scores come after settle_scores.
__device__ __forceinline__ float max3(float a, float b, float c) {
  float r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(r) : "v"(a), "v"(b), "v"(c));
  return r;
}
__device__ __forceinline__ float tile_max(const f32x16 (&v)[4]) {
  // 64 -> 22 -> 8 -> 3 -> 1
  float a[22], b[8], c[3];
#pragma unroll
  for (int i = 0; i < 21; ++i) {
    const int e0 = 3 * i, e1 = 3 * i + 1, e2 = 3 * i + 2;
    a[i] = max3(v[e0 >> 4][e0 & 15], v[e1 >> 4][e1 & 15], v[e2 >> 4][e2 & 15]);
  }
  a[21] = v[3][15];
#pragma unroll
  for (int i = 0; i < 7; ++i) b[i] = max3(a[3 * i], a[3 * i + 1], a[3 * i + 2]);
  b[7] = a[21];
  c[0] = max3(b[0], b[1], b[2]);
  c[1] = max3(b[3], b[4], b[5]);
  c[2] = max3(b[6], b[7], b[7]);
  return max3(c[0], c[1], c[2]);
}
__device__ __forceinline__ float tile_sum(const f32x16 (&v)[4]) {
  float a[16];
#pragma unroll
  for (int i = 0; i < 16; ++i) a[i] = (v[0][i] + v[1][i]) + (v[2][i] + v[3][i]);
#pragma unroll
  for (int w = 8; w >= 1; w >>= 1)
#pragma unroll
    for (int i = 0; i < w; ++i) a[i] = a[i] + a[i + w];
  return a[0];
}

// Two waves per SIMD, three for fp8 at d = 64 (163 VGPRs, 32 KB of LDS per
// workgroup: three workgroups fit a CU, and the third wave hides more of the
// VALU latency in that VALU-bound case).
template <int DT, int D, bool CAUSAL, int MODE, bool PROBE, bool CMP>
__global__ __launch_bounds__(MAX_THREADS) __attribute__((amdgpu_waves_per_eu(2, (DT == DT_FP8 && D == 64) ? 3 : 2))) void
attn_fwd_kernel(Params p) {
  using C = Cfg<DT, D, CMP>;
  constexpr int NW = C::NW, BR = C::BR;
  // K and V tiles, each double-buffered, or single-buffered: compact d = 128,
  // and the lattice weights at FP8 d = 128 (measured at causal and
  // non-causal 8K: H15 +1.7..2.4% single-buffered, the exact control
  // -0.7%, so the control keeps two buffers)
  constexpr int NSTAGE = (DT == DT_FP8 && D == 128 && mode_lattice(MODE)) ? 1 : C::NSTAGE;
  static_assert(NSTAGE == 2 || MODE != MODE_ROWMAX_POT, "the Rowmax-PoT first pass double-buffers K");
  __shared__ __attribute__((aligned(16))) uint8_t smem[NSTAGE * C::BUF];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int i32 = lane & 31;
  const int g = lane >> 5;
  const int G4 = lane >> 4, L16 = lane & 15;

  int qb, b, h;
  map_block(p, blockIdx.x, qb, b, h);
  const int S = p.S;
  const int hk = h / p.G;
  const int q0 = qb * BR;
  const int qw0 = q0 + wave * WROWS;
  const int qrow = qw0 + i32;
  const bool wave_live = qw0 < S;
  const int last_key = CAUSAL ? min(q0 + BR - 1, S - 1) : S - 1;
  const int ntiles = last_key / BC + 1;
  const float off = DT == DT_FP8 ? 8.0f : 0.0f;

  const size_t kv_head = (size_t)(b * p.Hkv + hk) * (size_t)S;
  const uint8_t* kg = p.k + kv_head * C::RB;
  const uint8_t* vg = p.v + kv_head * C::RB;
  const size_t q_head = (size_t)(b * p.Hq + h) * (size_t)S;

  // ---- Q block in registers (MFMA B operand: lane holds row i32, k-half g);
  // loaded through LDS below (stage_q, read_q)
  constexpr int NKQ = DT == DT_BF16 ? D / 16 : D / 64;
  bf16x8 qb16[DT == DT_BF16 ? NKQ : 1];
  i32x8 qf8[DT == DT_FP8 ? NKQ : 1];

  // ---- staging: every wave copies WAVE_LOADS x 1 KB of a K or V tile
  // straight into LDS.  LDS slot s (16 bytes) of a tile holds row s / NCH,
  // chunk (s % NCH) ^ swizzle(row).  Buffer (not global) loads are used so
  // that the compiler's wait counting keeps LDS reads pipelined while these
  // copies are in flight.  One head's rows span S * RB < 2^31 bytes.  Tile t
  // uses K buffer t % 2 and V buffer t % 2.
  const __amdgpu_buffer_rsrc_t krsrc = __builtin_amdgcn_make_buffer_rsrc((void*)kg, (short)0, S * C::RB, BUF_DWORD3);
  const __amdgpu_buffer_rsrc_t vrsrc = __builtin_amdgcn_make_buffer_rsrc((void*)vg, (short)0, S * C::RB, BUF_DWORD3);
  auto kbuf = [&](int t) { return smem + (t & 1) * C::BUF; };
  auto vbuf = [&](int t) { return smem + (t & 1) * C::BUF + C::TILE; };
  // Every wave copies its WAVE_LOADS 1 KB blocks of a tile.  The lane's byte
  // offset inside the tile is the same for every tile, so it is computed
  // once; a tile then adds only the scalar offset of its first row.  Rows at
  // or beyond S (the ragged last tile) lie outside the resource's
  // num_records = S * RB: the hardware range check (on the sum of both
  // offsets, per dword) reads them as zero without touching memory, and
  // those keys are masked.  The wave index is scalar, so the LDS
  // destinations (M0) are too.
  // (The addresses handed to the LDS-copy builtin are named variables: with
  // an arithmetic expression in those arguments the host side of this
  // compiler drops the kernels' launch stubs without a diagnostic.)
  constexpr int WAVE_LOADS = C::CHUNKS / (NW * 64);
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);
  uint32_t koff_c[WAVE_LOADS], voff_c[WAVE_LOADS];
#pragma unroll
  for (int c = 0; c < WAVE_LOADS; ++c) {
    const int slot = (c * NW + wave) * 64 + lane;
    const int row = slot / C::NCH, pch = slot % C::NCH;
    koff_c[c] = (uint32_t)(row * C::RB + ((pch ^ k_swz<DT, D>(row)) << 4));
    voff_c[c] = (uint32_t)(row * C::RB + ((pch ^ v_swz<DT, D>(row)) << 4));
  }
  auto stage = [&](int t, uint8_t* dst, const __amdgpu_buffer_rsrc_t& rsrc,
                   const uint32_t (&off_c)[WAVE_LOADS]) __attribute__((always_inline)) {
    const uint32_t soff = (uint32_t)(t * BC) * C::RB;
#pragma unroll
    for (int c = 0; c < WAVE_LOADS; ++c) {
      const uint32_t voff = off_c[c];
      uint8_t* ldst = dst + (c * NW + wave_s) * 1024;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, LDS_PTR(void, ldst), 16, voff, soff, 0, 0);
    }
  };
  auto stage_k = [&](int t) { stage(t, kbuf(t), krsrc, koff_c); };
  auto stage_v = [&](int t) { stage(t, vbuf(t), vrsrc, voff_c); };

  // ---- Q through LDS: each wave copies its own 32 rows with the same
  // direct loads (16 contiguous bytes per lane, so each load covers whole
  // rows; rows at or beyond S read as zero), into a region the first K/V
  // copies do not touch (the V buffer when single-buffered, else the second
  // buffer), chunks swizzled as K's so that the operand reads, one chunk of
  // 32 rows per instruction like K's, spread over the banks.  Every wave
  // reads its operands before any wave copies into that region again (a
  // barrier after read_q).
  constexpr int QBYTES = WROWS * C::RB;
  constexpr int QREGION = NSTAGE == 1 ? C::TILE : C::BUF;
  static_assert(QBYTES % 1024 == 0 && QREGION + NW * QBYTES <= NSTAGE * C::BUF, "Q staging layout");
  const __amdgpu_buffer_rsrc_t qrsrc =
      __builtin_amdgcn_make_buffer_rsrc((void*)(p.q + q_head * C::RB), (short)0, S * C::RB, BUF_DWORD3);
  uint8_t* const qreg = smem + QREGION + wave_s * QBYTES;
  auto stage_q = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < QBYTES / 1024; ++c) {
      const int slot = c * 64 + lane;
      const int row = slot / C::NCH, pch = slot % C::NCH;
      // (unsigned: rows past S may take the offset past 2^31, where the
      // range check still reads zero)
      const uint32_t voff = (uint32_t)(qw0 + row) * (uint32_t)C::RB + (uint32_t)((pch ^ k_swz<DT, D>(row)) << 4);
      uint8_t* ldst = qreg + c * 1024;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(qrsrc, LDS_PTR(void, ldst), 16, voff, 0, 0, 0);
    }
  };
  auto read_q = [&]() __attribute__((always_inline)) {
    const uint8_t* const qrow_l = qreg + i32 * C::RB;
    const int qswz = k_swz<DT, D>(i32);
    if constexpr (DT == DT_BF16) {
#pragma unroll
      for (int kk = 0; kk < NKQ; ++kk) qb16[kk] = *(const bf16x8*)(qrow_l + (((2 * kk + g) ^ qswz) << 4));
    } else {
#pragma unroll
      for (int kk = 0; kk < NKQ; ++kk) {
        const i32x4 lo = *(const i32x4*)(qrow_l + (((4 * kk + 2 * g) ^ qswz) << 4));
        const i32x4 hi = *(const i32x4*)(qrow_l + (((4 * kk + 2 * g + 1) ^ qswz) << 4));
        qf8[kk] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
    }
  };

  // ---- running state (this lane's query row; lanes i and i^32 agree on m)
  constexpr int NDB = D / 32;  // 32-column blocks of O^T
  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = f32x16{0.0f};
  float m_run = -INFINITY;
  float l_part = 0.0f;  // this lane's share of the row sum
  // scores, then weights, of the current tile; accumulator value j of block
  // kb holds key 32 kb + 8 (j/4) + 4 g + j%4 of the tile
  f32x16 sacc[4];
  // P of the current tile in the operand type (the MFMA B operand of PV)
  bf16x8 pb[DT == DT_BF16 ? 8 : 1];
  i32x8 pf[DT == DT_FP8 ? 2 : 1];
  // lattice modes: the weights as BF16 pairs, word q of block kb holding keys
  // 2q and 2q + 1 of sacc[kb]
  uint32_t wpk[4][8];
  // FP8 finishes the second half of the tile's P (keys 64..127)
  // between the PV MFMAs of the first half (MFMA i covers block db = i % NDB
  // of O^T and key half i / NDB), which do not depend on it, so
  // that the wave's own VALU work runs while its matrix core is busy; the
  // row sum's partial sums then stay open across the PV product (exact
  // mode: the two halves in lch; lattice modes: eight dot2 chains in lch8,
  // one per word index, none longer than four)
  constexpr bool SPLIT = DT == DT_FP8 && MODE != MODE_ROWMAX_POT;
  float lch[2];
  float lch8[8];
  float nb1_split = 0.0f;  // exact mode: the exponent bias of the open tile

  // ---- S^T = K Q^T for the 128 keys of a tile (4 blocks of 32 keys).
  // MFMA i covers (kk = i / 4, kb = i % 4).  Its K operand is read from LDS
  // QK_AHEAD MFMAs in advance into a ring of registers, and the schedule keeps
  // that order, so each MFMA finds its operand loaded.
  auto qk = [&](const uint8_t* kl) __attribute__((always_inline)) {
    const int krow_off = i32 * C::RB;
    const int kswz = k_swz<DT, D>(i32);  // == k_swz(kb * 32 + i32)
    constexpr int NQK = 4 * NKQ;
    if constexpr (DT == DT_BF16) {
      auto ldk = [&](int i) {
        const uint8_t* rowp = kl + (i & 3) * 32 * C::RB + krow_off;
        return *(const bf16x8*)(rowp + (((2 * (i >> 2) + g) ^ kswz) << 4));
      };
      bf16x8 ring[QK_AHEAD + 1];
#pragma unroll
      for (int i = 0; i < QK_AHEAD; ++i) ring[i] = ldk(i);
      __builtin_amdgcn_sched_barrier(0);  // the prologue reads go first
#pragma unroll
      for (int i = 0; i < NQK; ++i) {
        const int kk = i >> 2, kb = i & 3;
        sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(ring[i % (QK_AHEAD + 1)], qb16[kk],
                                                           kk == 0 ? f32x16{0.0f} : sacc[kb], 0, 0, 0);
        if (i + QK_AHEAD < NQK) ring[(i + QK_AHEAD) % (QK_AHEAD + 1)] = ldk(i + QK_AHEAD);
      }
#pragma unroll
      for (int i = 0; i < NQK; ++i) {
        __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
        if (i + QK_AHEAD < NQK) __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 1, 0);
      }
    } else {
      auto ldk = [&](int i) {
        const int kk = i >> 2;
        const uint8_t* rowp = kl + (i & 3) * 32 * C::RB + krow_off;
        const i32x4 lo = *(const i32x4*)(rowp + (((4 * kk + 2 * g) ^ kswz) << 4));
        const i32x4 hi = *(const i32x4*)(rowp + (((4 * kk + 2 * g + 1) ^ kswz) << 4));
        return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      };
      i32x8 ring[QK_AHEAD + 1];
#pragma unroll
      for (int i = 0; i < QK_AHEAD; ++i) ring[i] = ldk(i);
      __builtin_amdgcn_sched_barrier(0);  // the prologue reads go first
#pragma unroll
      for (int i = 0; i < NQK; ++i) {
        const int kk = i >> 2, kb = i & 3;
        sacc[kb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
            ring[i % (QK_AHEAD + 1)], qf8[kk], kk == 0 ? f32x16{0.0f} : sacc[kb], 0, 0, 0, 0, 0, 0);
        if (i + QK_AHEAD < NQK) ring[(i + QK_AHEAD) % (QK_AHEAD + 1)] = ldk(i + QK_AHEAD);
      }
#pragma unroll
      for (int i = 0; i < NQK; ++i) {
        __builtin_amdgcn_sched_group_barrier(SG_MFMA, 1, 0);
        if (i + QK_AHEAD < NQK) __builtin_amdgcn_sched_group_barrier(SG_DS_READ, 2, 0);
      }
    }
  };

  // ---- O^T += V^T P^T for the tile whose V sits at vl and whose P is in
  // pb/pf.  The V^T operands are read from LDS PV_AHEAD MFMAs ahead into a
  // ring of registers: pv_begin(vl) sets the lane's addresses and issues the
  // first PV_AHEAD reads (early, so that their latency hides behind the
  // softmax), pv_finish() issues the MFMAs and the remaining reads.  No
  // other LDS access may come between the two (the waits count reads).
  //
  // bf16: lane (d = i32 + 32 db, half g) needs keys 16 ks + 8 (r/4) + 4 g +
  // r%4 (r = 0..7): two 4-key transposing reads; lane L16 of a 16-lane group
  // addresses row 4 g + L16/4 (+8), columns 16 (G4%2) + 4 (L16%4) .. +3 of
  // the 32-column block.  MFMA i covers (db = i / 8, ks = i % 8).
  // fp8: lane (d = i32 + 32 db, half g) needs, for byte r = 8 rd + e, key
  // 32 (2 t2 + rd/2) + 16 (rd%2) + 8 (e/4) + 4 g + e%4: four 8-key
  // transposing reads; lane L16 of a 16-lane group addresses row vrow = base
  // + 8 (L16/8) + (L16/2)%4, columns d0 + 8 (L16%2) .. +7.  MFMA i covers
  // (db = i / 2, t2 = i % 2).
  // In both, the swizzle of the rows a lane reads equals that of vrow, so
  // only the block db moves the lane's address; the key offset is an
  // immediate.
  constexpr int NPV = DT == DT_BF16 ? NDB * 8 : NDB * 2;
  using VOp = std::conditional_t<DT == DT_BF16, bf16x8, i32x8>;
  VOp vring[PV_AHEAD + 1];
  uint32_t vbase[NDB];
  auto ldv = [&](auto ic) -> VOp {
    constexpr int i = decltype(ic)::value;
    if constexpr (DT == DT_BF16) {
      const i32x2v lo = ds_read_tr16<(16 * (i & 7)) * C::RB>(vbase[i >> 3]);
      const i32x2v hi = ds_read_tr16<(16 * (i & 7) + 8) * C::RB>(vbase[i >> 3]);
      return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3));
    } else {
      constexpr int t2 = SPLIT ? i / NDB : i & 1;
      const uint32_t a = vbase[SPLIT ? i % NDB : i >> 1];
      const i32x2v p0 = ds_read_tr8<(64 * t2) * C::RB>(a);
      const i32x2v p1 = ds_read_tr8<(64 * t2 + 16) * C::RB>(a);
      const i32x2v p2 = ds_read_tr8<(64 * t2 + 32) * C::RB>(a);
      const i32x2v p3 = ds_read_tr8<(64 * t2 + 48) * C::RB>(a);
      const i32x4 lo = __builtin_shufflevector(p0, p1, 0, 1, 2, 3);
      const i32x4 hi = __builtin_shufflevector(p2, p3, 0, 1, 2, 3);
      return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    }
  };
  auto pv_begin = [&](const uint8_t* vl) __attribute__((always_inline)) {
    const uint32_t vla = (uint32_t)(size_t)LDS_PTR(const uint8_t, vl);
    if constexpr (DT == DT_BF16) {
      const int vrow = 4 * (G4 >> 1) + (L16 >> 2);
      const int vcolb = (16 * (G4 & 1) + 4 * (L16 & 3)) * 2;
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const int cb = 64 * db + vcolb;
        vbase[db] = vla + vrow * C::RB + (((cb >> 4) ^ v_swz<DT, D>(vrow)) << 4) + (cb & 15);
      }
    } else {
      const int vrow = 4 * (G4 >> 1) + 8 * (L16 >> 3) + ((L16 >> 1) & 3);
      const int vcol = 16 * (G4 & 1) + 8 * (L16 & 1);
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const int cb = 32 * db + vcol;
        vbase[db] = vla + vrow * C::RB + (((cb >> 4) ^ v_swz<DT, D>(vrow)) << 4) + (cb & 15);
      }
    }
    static_for<0, PV_AHEAD>([&](auto ic) { vring[decltype(ic)::value] = ldv(ic); });
  };
  // ---- split P (FP8 lattice modes): part c (0..3) of the second half packs
  // words 4 (c % 2) .. +3 of block 2 + c / 2, converts them to P words 2c and
  // 2c + 1 of pf[1] and adds them to the row sum's chains
  auto finish_half = [&](auto cc) __attribute__((always_inline)) {
    if constexpr (SPLIT && !mode_lattice(MODE)) {
      // exact mode: part c takes values 8 (c % 2) .. +7 of block 2 + c / 2
      // through exp2, into P words 2c and 2c + 1, and sums them
      constexpr int c = decltype(cc)::value;
      constexpr int kb = 2 + (c >> 1), j0 = 8 * (c & 1);
#pragma unroll
      for (int j = j0; j < j0 + 8; ++j)
        sacc[kb][j] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kb][j], p.c1, nb1_split));
#pragma unroll
      for (int w = 0; w < 2; ++w) {
        const int jw = j0 + 4 * w;
        uint32_t word = __float_as_uint(sacc[kb][jw]);
        word = __builtin_amdgcn_cvt_pk_fp8_f32(sacc[kb][jw], sacc[kb][jw + 1], word, false);
        word = __builtin_amdgcn_cvt_pk_fp8_f32(sacc[kb][jw + 2], sacc[kb][jw + 3], word, true);
        pf[1][2 * c + w] = (int)word;
      }
      const float s8 = ((sacc[kb][j0] + sacc[kb][j0 + 1]) + (sacc[kb][j0 + 2] + sacc[kb][j0 + 3])) +
                       ((sacc[kb][j0 + 4] + sacc[kb][j0 + 5]) + (sacc[kb][j0 + 6] + sacc[kb][j0 + 7]));
      if constexpr ((c & 1) == 0) lch[c >> 1] = s8;
      else lch[c >> 1] += s8;
      if constexpr (c == 3) l_part += lch[0] + lch[1];
    } else if constexpr (SPLIT) {
      constexpr int c = decltype(cc)::value;
      constexpr int kb = 2 + (c >> 1), q0 = 4 * (c & 1);
#pragma unroll
      for (int q = q0; q < q0 + 4; ++q)
        wpk[kb][q] = sq_pack<MODE>(__float_as_uint(sacc[kb][2 * q]), __float_as_uint(sacc[kb][2 * q + 1]));
#pragma unroll
      for (int w = 0; w < 2; ++w) {
        i16x2 word = __builtin_bit_cast(i16x2, wpk[kb][q0 + 2 * w]);
        word = __builtin_amdgcn_cvt_scalef32_pk_fp8_bf16(word, __builtin_bit_cast(bf16x2, wpk[kb][q0 + 2 * w]), 1.0f,
                                                         false);
        word = __builtin_amdgcn_cvt_scalef32_pk_fp8_bf16(word, __builtin_bit_cast(bf16x2, wpk[kb][q0 + 2 * w + 1]),
                                                         1.0f, true);
        pf[1][2 * c + w] = __builtin_bit_cast(int, word);
      }
#pragma unroll
      for (int q = q0; q < q0 + 4; ++q) lch8[q] = dot2_ones(wpk[kb][q], lch8[q]);
      if constexpr (c == 3)
        l_part += ((lch8[0] + lch8[1]) + (lch8[2] + lch8[3])) + ((lch8[4] + lch8[5]) + (lch8[6] + lch8[7]));
    }
  };
  auto pv_finish = [&]() __attribute__((always_inline)) {
    // reads per operand
    constexpr int RPO = DT == DT_BF16 ? 2 : 4;
    static_for<0, NPV>([&](auto ic) {
      constexpr int i = decltype(ic)::value;
      // the reads of the PV_AHEAD - 1 later operands may still be in flight
      lds_wait<RPO * (i + PV_AHEAD <= NPV ? PV_AHEAD - 1 : NPV - 1 - i)>(vring[i % (PV_AHEAD + 1)]);
      if constexpr (DT == DT_BF16)
        oacc[i >> 3] =
            __builtin_amdgcn_mfma_f32_32x32x16_bf16(vring[i % (PV_AHEAD + 1)], pb[i & 7], oacc[i >> 3], 0, 0, 0);
      else {
        constexpr int db = SPLIT ? i % NDB : i >> 1, t2 = SPLIT ? i / NDB : i & 1;
        static_assert(db < NDB && t2 < 2, "PV operand index");
        oacc[db] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(vring[i % (PV_AHEAD + 1)], pf[t2], oacc[db], 0, 0,
                                                                   0, 0, 0, 0);
      }
      // each MFMA issues as soon as its operand is in (not after later reads)
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (i + PV_AHEAD < NPV)
        vring[(i + PV_AHEAD) % (PV_AHEAD + 1)] = ldv(std::integral_constant<int, i + PV_AHEAD>{});
      if constexpr (SPLIT && i < NDB) {
        // parts 4i/NDB .. 4(i+1)/NDB - 1 run while MFMA i executes; MFMAs
        // NDB .. 2 NDB - 1 read what they write
        static_for<4 * i / NDB, 4 * (i + 1) / NDB>([&](auto cc) { finish_half(cc); });
        __builtin_amdgcn_sched_barrier(0);
      }
    });
  };

  // ---- masked keys (causal diagonal, ragged tail) of tile t get score -inf;
  // returns whether the tile needed masking
  auto mask_scores = [&](int t) __attribute__((always_inline)) {
    const int kt0 = t * BC;
    const bool need_mask = (CAUSAL && kt0 + BC - 1 > qw0) || (kt0 + BC > S);
    if (need_mask) {
      const int lim = (CAUSAL ? min(qrow, S - 1) : S - 1) - kt0 - 4 * g;
      mask_beyond(sacc, lim, -INFINITY);
    }
    return need_mask;
  };

  // ---- the probe variant writes tile t's weights and P for its probed rows
  auto probe_weights = [&](int t) __attribute__((always_inline)) {
    if constexpr (PROBE) {
      const int kt0 = t * BC;
      if (b == p.pb && h == p.ph && qrow >= p.prow0 && qrow < p.prow0 + p.pnrows) {
        const size_t rbase = (size_t)(qrow - p.prow0) * S;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int key = kt0 + kb * 32 + 8 * (j >> 2) + 4 * g + (j & 3);
            if (key < S) {
              uint32_t bits;
              if constexpr (DT == DT_BF16) {
                // read the bf16 bits through a 32-bit view of the operand
                const u32x4 pw = __builtin_bit_cast(u32x4, pb[2 * kb + (j >> 3)]);
                bits = (pw[(j & 7) >> 1] >> (16 * (j & 1))) & 0xFFFFu;
              } else {
                bits = ((uint32_t)pf[kb >> 1][4 * (kb & 1) + (j >> 2)] >> (8 * (j & 3))) & 0xFFu;
              }
              p.w_out[rbase + key] =
                  mode_lattice(MODE) ? __uint_as_float(((wpk[kb][j >> 1] >> (16 * (j & 1))) & 0xFFFFu) << 16)
                                     : sacc[kb][j];
              p.p_out[rbase + key] = bits;
            }
          }
      }
    }
  };

  // ---- the scores of tile t become weights, the running state moves, and P
  // is left in pb/pf for the PV product
  auto softmax_tile = [&](int t, const uint8_t* vl) __attribute__((always_inline)) {
    const int kt0 = t * BC;

    // masking: causal diagonal and the ragged tail only
    const bool need_mask = mask_scores(t);

    const bool probe_row = PROBE && b == p.pb && h == p.ph && qrow >= p.prow0 && qrow < p.prow0 + p.pnrows;
    if constexpr (PROBE) {
      if (probe_row) {
        const size_t rbase = (size_t)(qrow - p.prow0) * S;
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int key = kt0 + kb * 32 + 8 * (j >> 2) + 4 * g + (j & 3);
            if (key < S) p.s_out[rbase + key] = sacc[kb][j];
          }
      }
    }

    // running maximum (threshold 0: moves to the maximum so far); Rowmax-PoT
    // keeps the whole-row maximum of its first pass
    float m_new = m_run;
    if constexpr (MODE != MODE_ROWMAX_POT) {
      const float mt = tile_max(sacc);
      float ma, mb;
      with_partner(mt, ma, mb);
      m_new = max3(m_run, ma, mb);
      if (DT == DT_BF16 && p.tau > 0.0f) {
        // conditional rescale (App. B.2; FP8 requires tau = 0): the anchor
        // moves only when the row's maximum grows by more than tau octaves
        // (FP32 test); per wave, when any real row of the wave does
        const float grow_by = (__builtin_fmaxf(ma, mb) - m_run) * p.c1;
        bool move = m_run == -INFINITY || grow_by > p.tau;
        if (p.tau_wave) move = __builtin_amdgcn_ballot_w64(move && qrow < S) != 0;
        if (!move) m_new = m_run;
      }
    }
    const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * p.c1);
    m_run = m_new;
    // the first V^T operands of this tile load while the weights are computed
    pv_begin(vl);

    // weights, in place over the scores (the lattice modes: as BF16 pairs)
    constexpr bool PACKED = mode_lattice(MODE);
    if constexpr (PACKED) {
      const float nbk = __builtin_fmaf(-m_new, p.ck, (float)(1 << mode_order(MODE)) * off);
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int j = 0; j < 16; ++j) sacc[kb][j] = __uint_as_float(sq_pre<MODE>(sacc[kb][j], p.ck, nbk));
      if (need_mask) {
        // masked keys carry weight 0 (the clamp alone would give 2^-126)
        if constexpr (mode_narrow(MODE)) {
          // their scores are -inf, so t = -inf here; every real t lies in
          // (0x1.8p23 - 2^15, 0x1.8p23 + 2^7), so one max lifts exactly the
          // masked keys to a value below all of them whose low half is the
          // masked-key lane value (v_max3: fmaxf would first canonicalise)
          const float lift = __uint_as_float(0x4B3F0000u | sq_masked<MODE>());
#pragma unroll
          for (int kb = 0; kb < 4; ++kb)
#pragma unroll
            for (int j = 0; j < 16; ++j) sacc[kb][j] = max3(sacc[kb][j], lift, lift);
        } else {
          const int lim = (CAUSAL ? min(qrow, S - 1) : S - 1) - kt0 - 4 * g;
          mask_beyond(sacc, lim, __uint_as_float(sq_masked<MODE>()));
        }
      }
#pragma unroll
      for (int kb = 0; kb < (SPLIT ? 2 : 4); ++kb)
#pragma unroll
        for (int q = 0; q < 8; ++q)
          wpk[kb][q] = sq_pack<MODE>(__float_as_uint(sacc[kb][2 * q]), __float_as_uint(sacc[kb][2 * q + 1]));
      if constexpr (SPLIT) {
        // eight chains, continued by finish_half
        l_part = l_part * alpha;
#pragma unroll
        for (int q = 0; q < 8; ++q) lch8[q] = dot2_ones(wpk[1][q], dot2_ones(wpk[0][q], 0.0f));
      } else {
        l_part = pair_sum(wpk, l_part * alpha);
      }
    } else {
      if constexpr (MODE == MODE_ROWMAX_POT) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int j = 0; j < 16; ++j) sacc[kb][j] = pot_weight(sacc[kb][j], m_new, p.c1);
        if (need_mask) {
          const int lim = (CAUSAL ? min(qrow, S - 1) : S - 1) - kt0 - 4 * g;
          mask_beyond(sacc, lim, 0.0f);
        }
      } else {
        const float nb1 = __builtin_fmaf(-m_new, p.c1, off);
#pragma unroll
        for (int kb = 0; kb < (SPLIT ? 2 : 4); ++kb)
#pragma unroll
          for (int j = 0; j < 16; ++j) sacc[kb][j] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kb][j], p.c1, nb1));
        nb1_split = nb1;
      }
      if constexpr (SPLIT) {
        // keys 0..63 now, 64..127 in finish_half
        float a[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) a[i] = sacc[0][i] + sacc[1][i];
#pragma unroll
        for (int w = 8; w >= 1; w >>= 1)
#pragma unroll
          for (int i = 0; i < w; ++i) a[i] = a[i] + a[i + w];
        l_part = l_part * alpha + a[0];
      } else {
        l_part = l_part * alpha + tile_sum(sacc);
      }
    }
    // skipping the rescale is exact when no row of the wave moved its max
    if (__builtin_amdgcn_ballot_w64(alpha != 1.0f) != 0) {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int j = 0; j < 16; ++j) oacc[db][j] *= alpha;
    }

    // P in the operand type
    if constexpr (DT == DT_BF16) {
#pragma unroll
      for (int ks = 0; ks < 8; ++ks) {
        if constexpr (PACKED) {
          const int kb = ks >> 1, q0 = 4 * (ks & 1);
          pb[ks] = __builtin_bit_cast(bf16x8, u32x4{wpk[kb][q0], wpk[kb][q0 + 1], wpk[kb][q0 + 2], wpk[kb][q0 + 3]});
        } else {
#pragma unroll
          for (int r = 0; r < 8; ++r) pb[ks][r] = (__bf16)sacc[ks >> 1][8 * (ks & 1) + r];
        }
      }
    } else {
#pragma unroll
      for (int t2 = 0; t2 < (SPLIT ? 1 : 2); ++t2)
#pragma unroll
        for (int w4 = 0; w4 < 8; ++w4) {
          const int kb = 2 * t2 + (w4 >> 2), j0 = 4 * (w4 & 3);
          if constexpr (PACKED) {
            // BF16 -> e4m3 with unit scale (the weights are exact in BF16);
            // the old value is fully overwritten by the two halves
            i16x2 word = __builtin_bit_cast(i16x2, wpk[kb][j0 / 2]);
            word = __builtin_amdgcn_cvt_scalef32_pk_fp8_bf16(word, __builtin_bit_cast(bf16x2, wpk[kb][j0 / 2]), 1.0f,
                                                             false);
            word = __builtin_amdgcn_cvt_scalef32_pk_fp8_bf16(word, __builtin_bit_cast(bf16x2, wpk[kb][j0 / 2 + 1]),
                                                             1.0f, true);
            pf[t2][w4] = __builtin_bit_cast(int, word);
          } else {
            // the old value is fully overwritten by the two halves
            uint32_t word = __float_as_uint(sacc[kb][j0]);
            word = __builtin_amdgcn_cvt_pk_fp8_f32(sacc[kb][j0], sacc[kb][j0 + 1], word, false);
            word = __builtin_amdgcn_cvt_pk_fp8_f32(sacc[kb][j0 + 2], sacc[kb][j0 + 3], word, true);
            pf[t2][w4] = (int)word;
          }
        }
    }
    if constexpr (!SPLIT) probe_weights(t);
  };

  // last tile holding a valid key for some row of this wave (-1: none)
  const int last_act = !wave_live ? -1 : (CAUSAL ? min(ntiles - 1, (qw0 + WROWS - 1) / BC) : ntiles - 1);
  if constexpr (MODE == MODE_ROWMAX_POT) {
    // ---- Rowmax-PoT anchors every weight at the whole-row maximum: a first
    // pass over the key tiles computes it (QK^T and the masked row max only)
    stage_q();
    stage_k(0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    read_q();
    __syncthreads();
    for (int t = 0; t < ntiles; ++t) {
      if (t + 1 < ntiles) stage_k(t + 1);
      if (t <= last_act) {
        __builtin_amdgcn_s_setprio(1);
        qk(kbuf(t));
        __builtin_amdgcn_s_setprio(0);
        settle_scores(sacc);
        mask_scores(t);
        const float mt = tile_max(sacc);
        float ma, mb;
        with_partner(mt, ma, mb);
        m_run = max3(m_run, ma, mb);
      }
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
    }
  }

  // ---- one tile per step: copy in the next tile, then QK^T, weights, PV.
  // Steps come in pairs so that each one's LDS buffers are fixed at compile
  // time and their addresses fold into the reads' immediate offsets.
  // Single-buffered tiles (compact d = 128): K(t + 1) is copied in once every
  // wave has read K(t), during the weights and PV of tile t, and V(t + 1)
  // once every wave has read V(t), during QK^T of tile t + 1; each wait for a
  // copy comes just before the barrier that makes it visible.
  auto step_single = [&](int t) __attribute__((always_inline)) {
    uint8_t* const kl = smem;
    uint8_t* const vl = smem + C::TILE;
    if (t <= last_act) {
      __builtin_amdgcn_s_setprio(1);
      qk(kl);
      __builtin_amdgcn_s_setprio(0);
      settle_scores(sacc);
    }
    // this wave's copy of V(t) has landed and its reads of K(t) are done
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (t + 1 < ntiles) stage(t + 1, kl, krsrc, koff_c);
    if (t <= last_act) {
      softmax_tile(t, vl);
      __builtin_amdgcn_s_setprio(1);
      pv_finish();
      __builtin_amdgcn_s_setprio(0);
      if constexpr (SPLIT) probe_weights(t);
    }
    // this wave's copy of K(t + 1) has landed and its reads of V(t) are done
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (t + 1 < ntiles) stage(t + 1, vl, vrsrc, voff_c);
  };
  auto step = [&](int t, auto par) __attribute__((always_inline)) {
    constexpr int P = decltype(par)::value;
    uint8_t* const kl = smem + P * C::BUF;
    uint8_t* const vl = kl + C::TILE;
    if (t + 1 < ntiles) {
      stage(t + 1, smem + (1 - P) * C::BUF, krsrc, koff_c);
      stage(t + 1, smem + (1 - P) * C::BUF + C::TILE, vrsrc, voff_c);
    }
    if (t <= last_act) {
      __builtin_amdgcn_s_setprio(1);
      qk(kl);
      __builtin_amdgcn_s_setprio(0);
      settle_scores(sacc);
      softmax_tile(t, vl);
      __builtin_amdgcn_s_setprio(1);
      pv_finish();
      __builtin_amdgcn_s_setprio(0);
      if constexpr (SPLIT) probe_weights(t);
    }
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
  };
  if constexpr (NSTAGE == 1) {
    stage_q();
    stage(0, smem, krsrc, koff_c);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    read_q();
    __syncthreads();
    stage(0, smem + C::TILE, vrsrc, voff_c);
    for (int t = 0; t < ntiles; ++t) step_single(t);
  } else {
    if constexpr (MODE != MODE_ROWMAX_POT) stage_q();
    stage_k(0);
    stage_v(0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if constexpr (MODE != MODE_ROWMAX_POT) {
      read_q();
      __syncthreads();
    }
    for (int t = 0; t < ntiles; t += 2) {
      step(t, std::integral_constant<int, 0>{});
      if (t + 1 < ntiles) step(t + 1, std::integral_constant<int, 1>{});
    }
  }

  // ---- epilogue: O = acc / l * v_descale (bf16), LSE
  if (!wave_live) return;
  float la, lb;
  with_partner(l_part, la, lb);
  const float l = la + lb;
  const float inv = p.vd / l;
  // O leaves through LDS, which is free once every wave has passed the last
  // barrier: the lanes write their four-column pieces into the wave's own
  // 32 x D block (16-byte chunks XOR-swizzled by row: the reads are free of
  // bank conflicts, the writes of rows r and r + 16 share banks) and read
  // back 16 contiguous bytes of a row, so that each global store covers
  // whole rows instead of 8 bytes in each of 32 rows
  constexpr int ORB = D * 2, ONC = ORB / 16;  // bytes and 16-byte chunks per O row
  static_assert(NW * WROWS * ORB <= NSTAGE * C::BUF, "O staging fits the tile buffers");
  uint8_t* const ost = smem + wave * (WROWS * ORB);
  auto oswz = [](int row) { return D == 128 ? (row & 15) : ((row >> 1) & 7); };
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int jq = 0; jq < 4; ++jq) {
      const __bf16 a0 = (__bf16)(oacc[db][4 * jq + 0] * inv);
      const __bf16 a1 = (__bf16)(oacc[db][4 * jq + 1] * inv);
      const __bf16 a2 = (__bf16)(oacc[db][4 * jq + 2] * inv);
      const __bf16 a3 = (__bf16)(oacc[db][4 * jq + 3] * inv);
      const uint32_t w01 = (uint32_t)__builtin_bit_cast(uint16_t, a0) |
                           ((uint32_t)__builtin_bit_cast(uint16_t, a1) << 16);
      const uint32_t w23 = (uint32_t)__builtin_bit_cast(uint16_t, a2) |
                           ((uint32_t)__builtin_bit_cast(uint16_t, a3) << 16);
      // columns 32 db + 8 jq + 4 g .. +3: chunk 4 db + jq, half g
      *(u32x2*)(ost + i32 * ORB + (((4 * db + jq) ^ oswz(i32)) << 4) + 8 * g) = u32x2{w01, w23};
    }
  // the wave reads what its other lanes wrote (LDS keeps a wave's order)
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  constexpr int RPI = 64 / ONC;  // rows per store
  const int rsub = lane / ONC, csub = lane % ONC;
  uint8_t* const obase = (uint8_t*)p.o + (q_head + qw0) * (size_t)ORB + csub * 16;
  u32x4 orows[WROWS / RPI];
#pragma unroll
  for (int k = 0; k < WROWS / RPI; ++k) {
    const int r = RPI * k + rsub;
    orows[k] = *(const u32x4*)(ost + r * ORB + ((csub ^ oswz(r)) << 4));
  }
  if (qw0 + WROWS <= S) {
#pragma unroll
    for (int k = 0; k < WROWS / RPI; ++k) *(u32x4*)(obase + (size_t)(RPI * k + rsub) * ORB) = orows[k];
  } else {
#pragma unroll
    for (int k = 0; k < WROWS / RPI; ++k)
      if (qw0 + RPI * k + rsub < S) *(u32x4*)(obase + (size_t)(RPI * k + rsub) * ORB) = orows[k];
  }
  if (p.lse && g == 0 && qrow < S)
    p.lse[q_head + qrow] = 0.69314718055994531f * (m_run * p.c1 + log2f(l) - off);
}

#if !H15_FP8_LATTICE_D128
// Probe support: pre-fill the probe buffers (s = -inf, w = 0, P = 0).
__global__ void probe_fill(float* s, float* w, uint32_t* pbits, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    s[i] = -INFINITY;
    w[i] = 0.0f;
    pbits[i] = 0u;
  }
}
#endif

template <int DT, int D, bool CAUSAL, int MODE, bool PROBE>
hipError_t launch_one(const Params& p, hipStream_t st) {
  const unsigned grid = (unsigned)(p.nqb * p.B * p.Hq);
  if constexpr (DT == DT_BF16 && MODE != MODE_ROWMAX_POT) {
    if (p.compact) {
      hipLaunchKernelGGL((attn_fwd_kernel<DT, D, CAUSAL, MODE, PROBE, true>), dim3(grid),
                         dim3(Cfg<DT, D, true>::NW * 64), 0, st, p);
      return hipGetLastError();
    }
  }
  if (p.compact) return hipErrorInvalidValue;  // offered for BF16 without Rowmax-PoT only
  hipLaunchKernelGGL((attn_fwd_kernel<DT, D, CAUSAL, MODE, PROBE, false>), dim3(grid), dim3(Cfg<DT, D>::NW * 64), 0,
                     st, p);
  return hipGetLastError();
}

#if H15_FP8_LATTICE_D128
template <bool CAUSAL, bool PROBE>
hipError_t launch_lattice128(const Params& p, int mode, hipStream_t st) {
  switch (mode) {
    case 1: return launch_one<DT_FP8, 128, CAUSAL, 1, PROBE>(p, st);
    case 2: return launch_one<DT_FP8, 128, CAUSAL, 2, PROBE>(p, st);
    case 3: return launch_one<DT_FP8, 128, CAUSAL, 3, PROBE>(p, st);
    case 4: return launch_one<DT_FP8, 128, CAUSAL, 4, PROBE>(p, st);
    case 5: return launch_one<DT_FP8, 128, CAUSAL, 5, PROBE>(p, st);
    case 6: return launch_one<DT_FP8, 128, CAUSAL, 6, PROBE>(p, st);
    default: return hipErrorInvalidValue;
  }
}
#else
template <int DT, int D, bool CAUSAL, bool PROBE>
hipError_t launch_mode(const Params& p, int mode, hipStream_t st) {
  if (mode == MODE_EXACT) return launch_one<DT, D, CAUSAL, MODE_EXACT, PROBE>(p, st);
  if constexpr (DT == DT_FP8 && D == 128) {
    // the FP8 lattice weights at d = 128 live in the other compilation of
    // this file
    return h15::launch_fwd_fp8_lattice128(p, CAUSAL, mode, st, PROBE);
  } else {
    switch (mode) {
      case 1: return launch_one<DT, D, CAUSAL, 1, PROBE>(p, st);
      case 3: return launch_one<DT, D, CAUSAL, 3, PROBE>(p, st);
      case 5: return launch_one<DT, D, CAUSAL, 5, PROBE>(p, st);
      default: break;
    }
    if constexpr (DT == DT_BF16) {
      if (mode == MODE_ROWMAX_POT) return launch_one<DT, D, CAUSAL, MODE_ROWMAX_POT, PROBE>(p, st);
    }
    // the narrow-clamp forms are only ever chosen for FP8
    if constexpr (DT == DT_FP8) {
      switch (mode) {
        case 2: return launch_one<DT, D, CAUSAL, 2, PROBE>(p, st);
        case 4: return launch_one<DT, D, CAUSAL, 4, PROBE>(p, st);
        case 6: return launch_one<DT, D, CAUSAL, 6, PROBE>(p, st);
        default: break;
      }
    }
    return hipErrorInvalidValue;
  }
}

template <int DT, int D, bool PROBE>
hipError_t launch_dt_d(const Params& p, int causal, int mode, hipStream_t st) {
  return causal ? launch_mode<DT, D, true, PROBE>(p, mode, st) : launch_mode<DT, D, false, PROBE>(p, mode, st);
}

template <bool PROBE>
hipError_t launch_any(const Params& p, int dtype, int d, int causal, int mode, hipStream_t st) {
  if (dtype == ATTN_BF16)
    return d == 128 ? launch_dt_d<DT_BF16, 128, PROBE>(p, causal, mode, st)
                    : launch_dt_d<DT_BF16, 64, PROBE>(p, causal, mode, st);
  return d == 128 ? launch_dt_d<DT_FP8, 128, PROBE>(p, causal, mode, st)
                  : launch_dt_d<DT_FP8, 64, PROBE>(p, causal, mode, st);
}

// ---------------------------------------------------------------------------
// Decode over a key/value cache: Sq query rows per head against Sk cached
// keys (bottom-right causal alignment), the keys cut into parts of
// split_keys keys that workgroups take in parallel.  Within a part the
// per-tile recurrence runs as in the forward kernel, with tiles starting at
// the part's first key and the running maximum starting at -inf; the parts'
// (m, l, O) then merge exactly (attn_decode_merge).  One part: the kernel
// normalises and writes O and LSE itself.
//
// One workgroup = 4 waves for one (batch, KV head, block of 32 query rows,
// part).  The 32 rows are the G * Sq query rows of the KV head's query heads
// (row r: head h = hkv G + r / Sq, position r % Sq), so the K/V tiles are read
// once for all of them.  Wave w computes the scores of keys 32w .. 32w + 31
// of each 128-key tile (one 32x32 block of S^T = K Q^T) and their share of
// PV; the tile maximum of each row is combined across the four waves through
// LDS, so every wave moves the same running maximum at every tile, and the
// waves' partial row sums and O accumulators, all relative to that maximum,
// are added up at the end.
//
// Decode reads the cache once and is bound by HBM, so the copies are laid
// out to keep as many bytes in flight as LDS allows: each wave loads only
// its own 32 keys, K straight into its MFMA operand registers (one tile
// ahead) and V into its own LDS slots (DEC_VSTAGES slots, so V of the next
// DEC_VSTAGES - 1 tiles is in flight); no barrier is needed for the copies,
// only the one per tile for the row maxima.  66 KB of LDS per group and at
// most 256 VGPRs per lane, so two groups share a CU (measured: with four
// times the V slots and one group per CU the per-tile chain of a lone wave
// per SIMD left FP8 decode 50% slower; with two groups FP8 +3% and BF16
// +11% against copies shared through double-buffered tiles).

constexpr int DEC_NW = 4;  // waves per decode workgroup (one 32-key block each)
template <int DT>
constexpr int dec_vstages() {
  return DT == DT_FP8 ? 4 : 2;
}

// s_waitcnt for vmcnt <= N only (gfx9 encoding: vmcnt in bits 3:0 and 15:14;
// expcnt 6:4 and lgkmcnt 11:8 at their maxima, so not waited for)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ void settle_block(f32x16& v) {
  // as settle_scores, for one block
  asm("s_nop 15\n\ts_nop 7" : "+v"(v));
}

template <int E = 0>
__device__ __forceinline__ void mask_beyond1(f32x16& v, int lim, float y) {
  if constexpr (E < 16) {
    v[E] = select_beyond<8 * (E >> 2) + (E & 3)>(lim, v[E], y);
    mask_beyond1<E + 1>(v, lim, y);
  }
}

__device__ __forceinline__ float block_max(const f32x16& v) {
  // 16 -> 6 -> 2 -> 1
  const float a0 = max3(v[0], v[1], v[2]), a1 = max3(v[3], v[4], v[5]), a2 = max3(v[6], v[7], v[8]);
  const float a3 = max3(v[9], v[10], v[11]), a4 = max3(v[12], v[13], v[14]);
  const float b0 = max3(a0, a1, a2), b1 = max3(a3, a4, v[15]);
  return max3(b0, b1, b1);
}

template <int DT, int D, bool CAUSAL, int MODE, bool PROBE>
__global__ __launch_bounds__(DEC_NW * 64) __attribute__((amdgpu_waves_per_eu(2, 2))) void attn_decode_kernel(
    DecParams p) {
  using C = Cfg<DT, D>;
  constexpr int NW = DEC_NW;
  constexpr int NSV = dec_vstages<DT>();
  constexpr int VSLOT = WROWS * C::RB;  // one wave's 32 V rows of a tile
  constexpr int NDB = D / 32;
  constexpr int NKQ = DT == DT_BF16 ? D / 16 : D / 64;
  constexpr int VLOADS = VSLOT / 1024;                   // 1 KB LDS copies per wave and tile
  constexpr int KLOADS = DT == DT_BF16 ? NKQ : 2 * NKQ;  // 16-byte K loads per lane and tile
  // loads issued after V(t) by the time tile t reads it, once every step
  // issues its K and V copies
  constexpr int VWAIT = (NSV - 1) * (KLOADS + VLOADS);
  static_assert(VSLOT % 1024 == 0 && (NSV & (NSV - 1)) == 0, "V slots");
  static_assert(NW * NDB * 16 * 64 * 4 <= NW * NSV * VSLOT, "the O reduction reuses the V slots");
  __shared__ __attribute__((aligned(16))) uint8_t smem[NW * NSV * VSLOT];
  __shared__ __attribute__((aligned(16))) float mx_lds[2][32][NW];
  __shared__ float l_lds[NW][64];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int i32 = lane & 31;
  const int g = lane >> 5;
  const int G4 = lane >> 4, L16 = lane & 15;

  int L = blockIdx.x;
  const int split = L % p.nsplit;
  L /= p.nsplit;
  const int rb = L % p.nrb;
  const int bkv = L / p.nrb;
  const int b = bkv / p.Hkv, hkv = bkv - b * p.Hkv;
  const int row = rb * WROWS + i32;
  const bool row_ok = row < p.R;
  const int rowc = min(row, p.R - 1);
  const int gq = rowc / p.Sq, iq = rowc - gq * p.Sq;
  const int h = hkv * p.G + gq;
  const size_t orow = (size_t)(b * p.Hq + h) * (size_t)p.Sq + (size_t)iq;
  const int Sk = p.Sk;
  const int limit = CAUSAL ? Sk - p.Sq + iq : Sk - 1;  // last key this row sees
  const int j0 = split * p.split_keys;
  const int j1 = min(j0 + p.split_keys, Sk);
  const int ntiles = (j1 - j0 + BC - 1) / BC;
  const float off = DT == DT_FP8 ? 8.0f : 0.0f;

  // ---- Q rows (MFMA B operand: lane holds row i32, k-half g)
  const uint8_t* qptr = p.q + orow * C::RB;
  bf16x8 qb16[DT == DT_BF16 ? NKQ : 1];
  i32x8 qf8[DT == DT_FP8 ? NKQ : 1];
  if constexpr (DT == DT_BF16) {
#pragma unroll
    for (int kk = 0; kk < NKQ; ++kk) qb16[kk] = *(const bf16x8*)(qptr + (16 * kk + 8 * g) * 2);
  } else {
#pragma unroll
    for (int kk = 0; kk < NKQ; ++kk) qf8[kk] = *(const i32x8*)(qptr + 64 * kk + 32 * g);
  }

  // ---- the part's K and V rows through buffer resources that start at the
  // part's first key and end at the cache length, so rows at or beyond Sk
  // read as zero (those keys are masked)
  const uint8_t* kg = p.k + ((size_t)bkv * (size_t)p.Sk_cap + (size_t)j0) * C::RB;
  const uint8_t* vg = p.v + ((size_t)bkv * (size_t)p.Sk_cap + (size_t)j0) * C::RB;
  const __amdgpu_buffer_rsrc_t krsrc =
      __builtin_amdgcn_make_buffer_rsrc((void*)kg, (short)0, (Sk - j0) * C::RB, BUF_DWORD3);
  const __amdgpu_buffer_rsrc_t vrsrc =
      __builtin_amdgcn_make_buffer_rsrc((void*)vg, (short)0, (Sk - j0) * C::RB, BUF_DWORD3);
  const int wave_s = __builtin_amdgcn_readfirstlane(wave);

  // K of this wave's 32 keys of tile t straight into the MFMA A operand
  // (lane: key 32 wave + i32; bf16: 16 bytes at 32 kk + 16 g of the row;
  // fp8: 32 bytes at 64 kk + 32 g)
  using KOp = std::conditional_t<DT == DT_BF16, bf16x8, i32x8>;
  const uint32_t krow = (uint32_t)((32 * wave + i32) * C::RB);
  auto load_k = [&](int t, KOp (&dst)[NKQ]) __attribute__((always_inline)) {
    const int soff = t * BC * C::RB;
#pragma unroll
    for (int kk = 0; kk < NKQ; ++kk) {
      if constexpr (DT == DT_BF16) {
        dst[kk] = __builtin_bit_cast(
            bf16x8, __builtin_amdgcn_raw_buffer_load_b128(krsrc, (int)(krow + 32 * kk + 16 * g), soff, 0));
      } else {
        const i32x4 lo = __builtin_bit_cast(
            i32x4, __builtin_amdgcn_raw_buffer_load_b128(krsrc, (int)(krow + 64 * kk + 32 * g), soff, 0));
        const i32x4 hi = __builtin_bit_cast(
            i32x4, __builtin_amdgcn_raw_buffer_load_b128(krsrc, (int)(krow + 64 * kk + 32 * g + 16), soff, 0));
        dst[kk] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      }
    }
  };
  // V of this wave's 32 keys of tile t into its LDS slot t % NSV: slot byte
  // s holds row s / RB with the forward kernel's chunk swizzle (the swizzle
  // depends on the row modulo 16, which the 32-row offset keeps)
  uint32_t voff_c[VLOADS];
#pragma unroll
  for (int c = 0; c < VLOADS; ++c) {
    const int slot = c * 64 + lane;
    const int r = slot / C::NCH, pch = slot % C::NCH;
    voff_c[c] = (uint32_t)(r * C::RB + ((pch ^ v_swz<DT, D>(r)) << 4));
  }
  auto vslot = [&](int t) { return smem + ((t & (NSV - 1)) * NW + wave_s) * VSLOT; };
  auto stage_v = [&](int t) __attribute__((always_inline)) {
    const uint32_t soff = (uint32_t)((t * BC + 32 * wave_s) * C::RB);
    uint8_t* const base = vslot(t);
#pragma unroll
    for (int c = 0; c < VLOADS; ++c) {
      const uint32_t voff = voff_c[c];
      uint8_t* ldst = base + c * 1024;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(vrsrc, LDS_PTR(void, ldst), 16, voff, soff, 0, 0);
    }
  };

  // ---- V^T operand addresses (as the forward kernel's, within this wave's
  // slot of 32 rows)
  uint32_t vbase[NDB];
  auto set_vbase = [&](const uint8_t* vl) __attribute__((always_inline)) {
    const uint32_t vla = (uint32_t)(size_t)LDS_PTR(const uint8_t, vl);
    if constexpr (DT == DT_BF16) {
      const int vrow = 4 * (G4 >> 1) + (L16 >> 2);
      const int vcolb = (16 * (G4 & 1) + 4 * (L16 & 3)) * 2;
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const int cb = 64 * db + vcolb;
        vbase[db] = vla + vrow * C::RB + (((cb >> 4) ^ v_swz<DT, D>(vrow)) << 4) + (cb & 15);
      }
    } else {
      const int vrow = 4 * (G4 >> 1) + 8 * (L16 >> 3) + ((L16 >> 1) & 3);
      const int vcol = 16 * (G4 & 1) + 8 * (L16 & 1);
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const int cb = 32 * db + vcol;
        vbase[db] = vla + vrow * C::RB + (((cb >> 4) ^ v_swz<DT, D>(vrow)) << 4) + (cb & 15);
      }
    }
  };

  f32x16 oacc[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db) oacc[db] = f32x16{0.0f};
  float m_run = -INFINITY;
  float l_part = 0.0f;
  const bool probe_row = PROBE && row_ok && b == p.pb && h == p.ph && iq == p.pi;

  // K(0) and V(0 .. NSV - 2) first; step t then issues K(t + 1) and
  // V(t + NSV - 1), in that order, before its own work
  KOp kreg[2][NKQ];
  load_k(0, kreg[0]);
  for (int s = 0; s < NSV - 1; ++s)
    if (s < ntiles) stage_v(s);
  auto step = [&](int t, KOp (&kc)[NKQ], KOp (&kn)[NKQ]) __attribute__((always_inline)) {
    if (t + 1 < ntiles) load_k(t + 1, kn);
    if (t + NSV - 1 < ntiles) stage_v(t + NSV - 1);
    const int kt0 = j0 + t * BC;    // first key of the tile
    const int kw0 = kt0 + 32 * wave;  // first key of this wave's block

    // ---- S^T block of this wave's 32 keys
    f32x16 sv;
    if constexpr (DT == DT_BF16) {
#pragma unroll
      for (int kk = 0; kk < NKQ; ++kk)
        sv = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kc[kk], qb16[kk], kk == 0 ? f32x16{0.0f} : sv, 0, 0, 0);
    } else {
#pragma unroll
      for (int kk = 0; kk < NKQ; ++kk)
        sv = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(kc[kk], qf8[kk], kk == 0 ? f32x16{0.0f} : sv, 0, 0, 0,
                                                             0, 0, 0);
    }
    settle_block(sv);

    // ---- masking: keys beyond the row's limit or the cache
    const bool need_mask = (CAUSAL && kt0 + BC - 1 > Sk - p.Sq) || (kt0 + BC > Sk);
    const int lim = limit - kw0 - 4 * g;
    if (need_mask) mask_beyond1(sv, lim, -INFINITY);
    if constexpr (PROBE) {
      if (probe_row) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int key = kw0 + 8 * (j >> 2) + 4 * g + (j & 3);
          if (key < Sk) p.s_out[key] = sv[j];
        }
      }
    }

    // ---- the tile maximum of each row, over the four waves' blocks
    {
      float ma, mb;
      with_partner(block_max(sv), ma, mb);
      if (g == 0) mx_lds[t & 1][i32][wave] = __builtin_fmaxf(ma, mb);
    }
    // (the two copies of mx_lds alternate, so a wave that runs ahead writes
    // the other one: every wave has read this one before the next barrier)
    __syncthreads();
    const f32x4 mx4 = *(const f32x4*)&mx_lds[t & 1][i32][0];
    const float m_new = max3(m_run, __builtin_fmaxf(mx4[0], mx4[1]), __builtin_fmaxf(mx4[2], mx4[3]));
    // a row that has seen no key yet keeps m = -inf, l = 0, O = 0
    const float alpha = m_new == -INFINITY ? 1.0f : __builtin_amdgcn_exp2f((m_run - m_new) * p.c1);
    const float m_use = m_new == -INFINITY ? 0.0f : m_new;
    m_run = m_new;

    // ---- weights (in place), row sum, P
    uint32_t wpk[8];
    constexpr bool PACKED = mode_lattice(MODE);
    if constexpr (PACKED) {
      const float nbk = __builtin_fmaf(-m_use, p.ck, (float)(1 << mode_order(MODE)) * off);
#pragma unroll
      for (int j = 0; j < 16; ++j) sv[j] = __uint_as_float(sq_pre<MODE>(sv[j], p.ck, nbk));
      if (need_mask) {
        if constexpr (mode_narrow(MODE)) {
          const float lift = __uint_as_float(0x4B3F0000u | sq_masked<MODE>());
#pragma unroll
          for (int j = 0; j < 16; ++j) sv[j] = max3(sv[j], lift, lift);
        } else {
          mask_beyond1(sv, lim, __uint_as_float(sq_masked<MODE>()));
        }
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) wpk[q] = sq_pack<MODE>(__float_as_uint(sv[2 * q]), __float_as_uint(sv[2 * q + 1]));
      float a0 = l_part * alpha, a1 = 0.0f;
#pragma unroll
      for (int q = 0; q < 8; q += 2) {
        a0 = dot2_ones(wpk[q], a0);
        a1 = dot2_ones(wpk[q + 1], a1);
      }
      l_part = a0 + a1;
    } else {
      const float nb1 = __builtin_fmaf(-m_use, p.c1, off);
#pragma unroll
      for (int j = 0; j < 16; ++j) sv[j] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[j], p.c1, nb1));
      float a[8];
#pragma unroll
      for (int i = 0; i < 8; ++i) a[i] = sv[i] + sv[i + 8];
#pragma unroll
      for (int w = 4; w >= 1; w >>= 1)
#pragma unroll
        for (int i = 0; i < w; ++i) a[i] = a[i] + a[i + w];
      l_part = l_part * alpha + a[0];
    }
    if (__builtin_amdgcn_ballot_w64(alpha != 1.0f) != 0) {
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int j = 0; j < 16; ++j) oacc[db][j] *= alpha;
    }

    // P in the operand type: bf16 as two 16-key operands; fp8 as one 64-key
    // operand whose other 32 keys (another wave's) carry P = 0
    bf16x8 pb2[2];
    i32x8 pf;
    if constexpr (DT == DT_BF16) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        if constexpr (PACKED) {
          pb2[ks] = __builtin_bit_cast(bf16x8, u32x4{wpk[4 * ks], wpk[4 * ks + 1], wpk[4 * ks + 2], wpk[4 * ks + 3]});
        } else {
#pragma unroll
          for (int r = 0; r < 8; ++r) pb2[ks][r] = (__bf16)sv[8 * ks + r];
        }
      }
    } else {
      int pw[4];
#pragma unroll
      for (int w4 = 0; w4 < 4; ++w4) {
        if constexpr (PACKED) {
          i16x2 word = __builtin_bit_cast(i16x2, wpk[2 * w4]);
          word = __builtin_amdgcn_cvt_scalef32_pk_fp8_bf16(word, __builtin_bit_cast(bf16x2, wpk[2 * w4]), 1.0f, false);
          word = __builtin_amdgcn_cvt_scalef32_pk_fp8_bf16(word, __builtin_bit_cast(bf16x2, wpk[2 * w4 + 1]), 1.0f,
                                                           true);
          pw[w4] = __builtin_bit_cast(int, word);
        } else {
          uint32_t word = __float_as_uint(sv[4 * w4]);
          word = __builtin_amdgcn_cvt_pk_fp8_f32(sv[4 * w4], sv[4 * w4 + 1], word, false);
          word = __builtin_amdgcn_cvt_pk_fp8_f32(sv[4 * w4 + 2], sv[4 * w4 + 3], word, true);
          pw[w4] = (int)word;
        }
      }
      if (wave & 1) pf = i32x8{0, 0, 0, 0, pw[0], pw[1], pw[2], pw[3]};
      else pf = i32x8{pw[0], pw[1], pw[2], pw[3], 0, 0, 0, 0};
    }
    if constexpr (PROBE) {
      if (probe_row) {
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const int key = kw0 + 8 * (j >> 2) + 4 * g + (j & 3);
          if (key < Sk && key <= limit) {
            uint32_t bits;
            if constexpr (DT == DT_BF16) {
              const u32x4 pw4 = __builtin_bit_cast(u32x4, pb2[j >> 3]);
              bits = (pw4[(j & 7) >> 1] >> (16 * (j & 1))) & 0xFFFFu;
            } else {
              bits = ((uint32_t)pf[4 * (wave & 1) + (j >> 2)] >> (8 * (j & 3))) & 0xFFu;
            }
            p.w_out[key] = mode_lattice(MODE) ? __uint_as_float(((wpk[j >> 1] >> (16 * (j & 1))) & 0xFFFFu) << 16)
                                              : sv[j];
            p.p_out[key] = bits;
          }
        }
      }
    }

    // ---- O^T += V^T P^T over this wave's keys, from its slot of V(t): this
    // wave's copy of V(t) has landed once at most VWAIT later loads are
    // outstanding (when every step so far issued its copies), or none is.
    // (The probe's stores also count as outstanding memory operations, so
    // the probe waits for all.)
    if (!PROBE && t >= NSV - 1 && t + NSV - 1 < ntiles) wait_vmcnt<VWAIT>();
    else wait_vmcnt<0>();
    set_vbase(vslot(t));
    if constexpr (DT == DT_BF16) {
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        i32x2v r0 = ds_read_tr16<0>(vbase[db]);
        i32x2v r1 = ds_read_tr16<8 * C::RB>(vbase[db]);
        i32x2v r2 = ds_read_tr16<16 * C::RB>(vbase[db]);
        i32x2v r3 = ds_read_tr16<24 * C::RB>(vbase[db]);
        lds_wait<0>(r0);
        lds_wait<0>(r1);
        lds_wait<0>(r2);
        lds_wait<0>(r3);
        const bf16x8 v0 = __builtin_bit_cast(bf16x8, __builtin_shufflevector(r0, r1, 0, 1, 2, 3));
        const bf16x8 v1 = __builtin_bit_cast(bf16x8, __builtin_shufflevector(r2, r3, 0, 1, 2, 3));
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v0, pb2[0], oacc[db], 0, 0, 0);
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(v1, pb2[1], oacc[db], 0, 0, 0);
      }
    } else {
      const i32x2v zero2 = {0, 0};
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        i32x2v r0 = ds_read_tr8<0>(vbase[db]);
        i32x2v r1 = ds_read_tr8<16 * C::RB>(vbase[db]);
        lds_wait<0>(r0);
        lds_wait<0>(r1);
        const i32x4 mine = __builtin_shufflevector(r0, r1, 0, 1, 2, 3);
        const i32x4 none = __builtin_shufflevector(zero2, zero2, 0, 1, 2, 3);
        const i32x8 vop = (wave & 1) ? __builtin_shufflevector(none, mine, 0, 1, 2, 3, 4, 5, 6, 7)
                                     : __builtin_shufflevector(mine, none, 0, 1, 2, 3, 4, 5, 6, 7);
        oacc[db] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(vop, pf, oacc[db], 0, 0, 0, 0, 0, 0);
      }
    }
  };
  // tiles in pairs, so that each step's K registers are fixed at compile time
  for (int t = 0; t < ntiles; t += 2) {
    step(t, kreg[0], kreg[1]);
    if (t + 1 < ntiles) step(t + 1, kreg[1], kreg[0]);
  }
  // every copy has landed and every wave is done with its V slots before the
  // slots are reused for the reduction
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();

  // ---- the four waves' partial sums: O^T blocks and row sums through LDS
  {
    float la, lb;
    with_partner(l_part, la, lb);
    l_lds[wave][lane] = la + lb;
    float* red = (float*)smem;  // [wave][db][j][lane]
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int j = 0; j < 16; ++j) red[((wave * NDB + db) * 16 + j) * 64 + lane] = oacc[db][j];
  }
  __syncthreads();
  if (!row_ok) return;
  const float l = (l_lds[0][lane] + l_lds[1][lane]) + (l_lds[2][lane] + l_lds[3][lane]);
  if (wave < NDB) {
    const int db = wave;
    const float* red = (const float*)smem;
    f32x16 osum;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      float acc = 0.0f;
#pragma unroll
      for (int w = 0; w < NW; ++w) acc += red[((w * NDB + db) * 16 + j) * 64 + lane];
      osum[j] = acc;
    }
    if (p.nsplit == 1) {
      const float inv = p.vd / l;
      uint16_t* orp = p.o + orow * (size_t)D;
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        const int col = 32 * db + 8 * jq + 4 * g;
        const __bf16 a0 = (__bf16)(osum[4 * jq + 0] * inv);
        const __bf16 a1 = (__bf16)(osum[4 * jq + 1] * inv);
        const __bf16 a2 = (__bf16)(osum[4 * jq + 2] * inv);
        const __bf16 a3 = (__bf16)(osum[4 * jq + 3] * inv);
        const uint32_t w01 = (uint32_t)__builtin_bit_cast(uint16_t, a0) |
                             ((uint32_t)__builtin_bit_cast(uint16_t, a1) << 16);
        const uint32_t w23 = (uint32_t)__builtin_bit_cast(uint16_t, a2) |
                             ((uint32_t)__builtin_bit_cast(uint16_t, a3) << 16);
        *(u32x2*)(orp + col) = u32x2{w01, w23};
      }
    } else {
      float* pop = p.part_o + (orow * (size_t)p.nsplit + (size_t)split) * (size_t)D;
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        const int col = 32 * db + 8 * jq + 4 * g;
        *(f32x4*)(pop + col) = f32x4{osum[4 * jq], osum[4 * jq + 1], osum[4 * jq + 2], osum[4 * jq + 3]};
      }
    }
  }
  if (wave == 0 && g == 0) {
    if (p.nsplit == 1) {
      if (p.lse) p.lse[orow] = 0.69314718055994531f * (m_run * p.c1 + log2f(l) - off);
    } else {
      *(f32x2*)(p.part_ml + (orow * (size_t)p.nsplit + (size_t)split) * 2) = f32x2{m_run, l};
    }
  }
}

struct MergeParams {
  const float* part_o;
  const float* part_ml;
  uint16_t* o;
  float* lse;
  int rows, nsplit;
  float c1, vd, off;
};

// The parts of each output row merged exactly: m = max m_p, f_p =
// 2^(c1 (m_p - m)) (0 for a part that saw no key), l = sum f_p l_p,
// O = sum f_p O_p / l * v_descale, LSE = ln2 (m c1 + log2 l - off).  One wave
// per row; lane j holds elements j * D / 64 .. of the row.
template <int D>
__global__ __launch_bounds__(256) void attn_decode_merge(MergeParams p) {
  constexpr int E = D / 64;
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  if (row >= p.rows) return;
  const float* ml = p.part_ml + (size_t)row * p.nsplit * 2;
  float m = -INFINITY;
  for (int s = 0; s < p.nsplit; ++s) m = __builtin_fmaxf(m, ml[2 * s]);
  float l = 0.0f;
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.0f;
  const float* po = p.part_o + (size_t)row * p.nsplit * D + lane * E;
  for (int s = 0; s < p.nsplit; ++s) {
    const float ms = ml[2 * s];
    const float f = ms == -INFINITY ? 0.0f : __builtin_amdgcn_exp2f((ms - m) * p.c1);
    l += f * ml[2 * s + 1];
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] += f * po[(size_t)s * D + e];
  }
  const float inv = p.vd / l;
  uint16_t* orp = p.o + (size_t)row * D + lane * E;
#pragma unroll
  for (int e = 0; e < E; ++e) orp[e] = __builtin_bit_cast(uint16_t, (__bf16)(acc[e] * inv));
  if (p.lse && lane == 0) p.lse[row] = 0.69314718055994531f * (m * p.c1 + log2f(l) - p.off);
}

template <int DT, int D, bool CAUSAL, int MODE, bool PROBE>
hipError_t launch_dec_one(const DecParams& p, hipStream_t st) {
  const unsigned grid = (unsigned)(p.B * p.Hkv * p.nrb * p.nsplit);
  hipLaunchKernelGGL((attn_decode_kernel<DT, D, CAUSAL, MODE, PROBE>), dim3(grid), dim3(DEC_NW * 64), 0, st, p);
  return hipGetLastError();
}

template <int DT, int D, bool CAUSAL, bool PROBE>
hipError_t launch_dec_mode(const DecParams& p, int mode, hipStream_t st) {
  switch (mode) {
    case MODE_EXACT: return launch_dec_one<DT, D, CAUSAL, MODE_EXACT, PROBE>(p, st);
    case 1: return launch_dec_one<DT, D, CAUSAL, 1, PROBE>(p, st);
    case 3: return launch_dec_one<DT, D, CAUSAL, 3, PROBE>(p, st);
    case 5: return launch_dec_one<DT, D, CAUSAL, 5, PROBE>(p, st);
    default: break;
  }
  if constexpr (DT == DT_FP8) {
    switch (mode) {
      case 2: return launch_dec_one<DT, D, CAUSAL, 2, PROBE>(p, st);
      case 4: return launch_dec_one<DT, D, CAUSAL, 4, PROBE>(p, st);
      case 6: return launch_dec_one<DT, D, CAUSAL, 6, PROBE>(p, st);
      default: break;
    }
  }
  return hipErrorInvalidValue;
}

template <bool PROBE>
hipError_t launch_dec_any(const DecParams& p, int dtype, int d, int causal, int mode, hipStream_t st) {
  if (dtype == ATTN_BF16) {
    if (d == 128)
      return causal ? launch_dec_mode<DT_BF16, 128, true, PROBE>(p, mode, st)
                    : launch_dec_mode<DT_BF16, 128, false, PROBE>(p, mode, st);
    return causal ? launch_dec_mode<DT_BF16, 64, true, PROBE>(p, mode, st)
                  : launch_dec_mode<DT_BF16, 64, false, PROBE>(p, mode, st);
  }
  if (d == 128)
    return causal ? launch_dec_mode<DT_FP8, 128, true, PROBE>(p, mode, st)
                  : launch_dec_mode<DT_FP8, 128, false, PROBE>(p, mode, st);
  return causal ? launch_dec_mode<DT_FP8, 64, true, PROBE>(p, mode, st)
                : launch_dec_mode<DT_FP8, 64, false, PROBE>(p, mode, st);
}

hipError_t launch_merge(const DecParams& dp, int dtype, int d, hipStream_t st) {
  MergeParams mp;
  mp.part_o = dp.part_o;
  mp.part_ml = dp.part_ml;
  mp.o = dp.o;
  mp.lse = dp.lse;
  mp.rows = dp.B * dp.Hq * dp.Sq;
  mp.nsplit = dp.nsplit;
  mp.c1 = dp.c1;
  mp.vd = dp.vd;
  mp.off = dtype == ATTN_FP8_E4M3 ? 8.0f : 0.0f;
  const unsigned grid = (unsigned)((mp.rows + 3) / 4);
  if (d == 128) hipLaunchKernelGGL(attn_decode_merge<128>, dim3(grid), dim3(256), 0, st, mp);
  else hipLaunchKernelGGL(attn_decode_merge<64>, dim3(grid), dim3(256), 0, st, mp);
  return hipGetLastError();
}

// Built-in workspace of attn_decode_noalloc: the parts' (m, l, O) of one
// decode call, for callers that cannot allocate.  Each GPU the library runs
// on holds its own copy until the process ends.  In host code the name is
// only a stand-in for the device address: the address each device uses is
// looked up once per device (scratch_address) and only that is passed on.
constexpr size_t SCRATCH_BYTES = (size_t)16 << 20;
static __device__ __align__(256) uint8_t scratch[SCRATCH_BYTES];

#endif  // !H15_FP8_LATTICE_D128

}  // namespace

namespace h15 {

#if H15_FP8_LATTICE_D128
hipError_t launch_fwd_fp8_lattice128(const Params& p, bool causal, int mode, hipStream_t st, bool probe) {
  if (probe) return causal ? launch_lattice128<true, true>(p, mode, st) : launch_lattice128<false, true>(p, mode, st);
  return causal ? launch_lattice128<true, false>(p, mode, st) : launch_lattice128<false, false>(p, mode, st);
}
#else
size_t scratch_capacity() { return SCRATCH_BYTES; }

int scratch_address(void* stream, void** ptr) {
  constexpr int MAX_DEVICES = 64;
  static std::mutex mu;
  static void* addr[MAX_DEVICES] = {};
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return 1;
  if (stream) {
    // the kernels run on the stream's device: its buffer is the one to use,
    // and it is looked up with the current device, so the two must agree
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice((hipStream_t)stream, &sdev) != hipSuccess) return 1;
    if (sdev != dev) return 2;
  }
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    // with the device current: this device's copy of the array
    void* a = nullptr;
    if (hipGetSymbolAddress(&a, HIP_SYMBOL(scratch)) != hipSuccess || !a) return 1;
    addr[dev] = a;
  }
  *ptr = addr[dev];
  return 0;
}

int launch_fwd(const Params& p, int dtype, int d, int causal, int mode, void* stream, bool probe) {
  hipStream_t st = (hipStream_t)stream;
  const hipError_t e = probe ? launch_any<true>(p, dtype, d, causal, mode, st)
                             : launch_any<false>(p, dtype, d, causal, mode, st);
  return e == hipSuccess ? 0 : 1;
}

int launch_probe_fill(float* s, float* w, uint32_t* pbits, size_t n, void* stream) {
  hipLaunchKernelGGL(probe_fill, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, (hipStream_t)stream, s, w, pbits,
                     n);
  return hipGetLastError() == hipSuccess ? 0 : 1;
}

int launch_decode(const DecParams& p, int dtype, int d, int causal, int mode, void* stream, bool probe) {
  hipStream_t st = (hipStream_t)stream;
  hipError_t e = probe ? launch_dec_any<true>(p, dtype, d, causal, mode, st)
                       : launch_dec_any<false>(p, dtype, d, causal, mode, st);
  if (e == hipSuccess && p.nsplit > 1) e = launch_merge(p, dtype, d, st);
  return e == hipSuccess ? 0 : 1;
}
#endif

}  // namespace h15
