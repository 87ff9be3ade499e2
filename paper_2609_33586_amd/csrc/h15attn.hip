// Fused attention forward for gfx950 (MI355X) with the softmax exponential
// either the hardware exp2 (control) or Rowmax-H15 (Sec. 5.2 Eq. (m-h15),
// App. B.1 "Implementation"), behind the C ABI declared in h15attn.h.
//
// Kernel structure (one workgroup = 8 wave64s = 256 query rows of one head):
//   * each wave keeps its 32 query rows of Q in VGPRs as the MFMA B operand;
//   * key tiles of 128 keys are staged HBM -> VGPR -> LDS, double-buffered:
//     the loads of tile t+1 are in flight while tile t is computed, and one
//     barrier per tile separates the buffers;
//   * scores are computed transposed, S^T = K Q^T, with 32x32 MFMAs (bf16
//     32x32x16, fp8 32x32x64): each lane then owns one query row and 64 of
//     the tile's 128 keys, so the row max and row sum are in-lane reductions
//     plus one exchange with lane ^ 32;
//   * the weights w are produced in VALU registers (hardware exp2, or the
//     H15 add/shift), converted to the MFMA operand type and used directly
//     as the B operand of O^T += V^T P^T: the MFMA contraction index is
//     mapped to keys so that the S accumulator layout is already the P
//     operand layout, with V read through the matching key order;
//   * V is read from LDS with ds_read_b64_tr_b16 (bf16) or stored transposed
//     in LDS at staging time (fp8).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "h15attn.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x4v __attribute__((__vector_size__(4 * sizeof(__bf16))));

constexpr int NW = 8;           // waves per workgroup
constexpr int WROWS = 32;       // query rows per wave
constexpr int BR = NW * WROWS;  // query rows per workgroup
constexpr int BC = 128;         // keys per tile (the running max moves once per tile)
constexpr int NTHREADS = NW * 64;
constexpr float H15_MAGIC = 12582912.0f;  // 0x4B400000 = 2^23 + 2^22
constexpr uint32_t ONE_BITS = 0x3F800000u;

enum { DT_BF16 = 0, DT_FP8 = 1 };
enum { MODE_EXACT = 0, MODE_H15 = 1 };

struct Params {
  const uint8_t* q;
  const uint8_t* k;
  const uint8_t* v;
  uint16_t* o;
  float* lse;
  int B, Hq, Hkv, S, G;
  float c1, c2, vd;
  int nqb;    // query blocks per head
  int remap;  // XCD-grouped workgroup order is valid for this shape
  // probe target (PROBE instantiations only)
  int pb, ph, prow0, pnrows;
  float* s_out;
  float* w_out;
  uint32_t* p_out;
};

template <int DT, int D>
struct Cfg {
  static constexpr int EB = DT == DT_BF16 ? 2 : 1;  // operand bytes
  static constexpr int RB = D * EB;                 // bytes per K/V row
  static constexpr int NCH = RB / 16;               // 16-byte chunks per row
  static constexpr int KT = BC * RB;                // K tile bytes
  static constexpr int VPITCH = BC + 16;            // fp8: bytes per V^T row (one d)
  static constexpr int VT = DT == DT_BF16 ? BC * RB : D * VPITCH;
  static constexpr int BUF = KT + VT;
  static constexpr int KCH = BC * NCH / NTHREADS;   // K chunks staged per thread
  static constexpr int VCH = DT == DT_BF16 ? KCH : 1;
  static constexpr int VSW = NCH >= 16 ? 4 : 2;     // bf16 V swizzle step
  static_assert(KCH >= 1, "tile too small for the staging layout");
};

// XOR swizzles of 16-byte chunks inside a row (bank spreading for the MFMA
// operand reads; the staging writes use the same map).
template <int DT, int D>
__device__ __forceinline__ int k_off(int row, int chunk) {
  using C = Cfg<DT, D>;
  return row * C::RB + ((chunk ^ (row % C::NCH)) << 4);
}
template <int DT, int D>
__device__ __forceinline__ int v_off(int row, int byte_in_row) {  // bf16 V, row-major
  using C = Cfg<DT, D>;
  const int chunk = byte_in_row >> 4;
  return row * C::RB + (((chunk ^ (C::VSW * (row & 3))) % C::NCH) << 4) + (byte_in_row & 15);
}
// fp8 V^T position of a key inside the tile: key = 32 blk + 8 m + 4 g + c is
// stored at 32 blk + 16 g + 4 m + c, so that the 16 keys one MFMA lane half
// multiplies are contiguous.
__device__ __forceinline__ int vt_pos(int key) {
  return (key & ~31) | ((key & 4) << 2) | ((key & 24) >> 1) | (key & 3);
}

__device__ __forceinline__ void map_block(const Params& p, int L, int& qb, int& b, int& h) {
  const int nbh = p.B * p.Hq;
  if (p.remap) {
    // Hardware workgroup ids go round-robin over the 8 XCDs (id mod 8).  Give
    // each XCD whole key/value-head groups, so the query heads that read the
    // same K/V share one L2, and walk query blocks longest-first.
    const int x = L & 7, j = L >> 3;
    const int per = nbh >> 3;
    const int qi = j / per, loc = j - qi * per;
    qb = p.nqb - 1 - qi;
    const int kvl = loc / p.G, gi = loc - kvl * p.G;
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

__device__ __forceinline__ float h15_weight(float s, float c2, float nb2) {
  // App. B.1: doubled exponent, clamp at -252, RNE add of 0x4B400000, shift
  // left by 22, add the bits of 1.0 (all modulo 2^32).
  float y = __builtin_fmaf(s, c2, nb2);
  y = __builtin_fmaxf(y, -252.0f);
  const float t = y + H15_MAGIC;
  return __uint_as_float((__float_as_uint(t) << 22) + ONE_BITS);
}

template <int DT, int D, bool CAUSAL, int MODE, bool PROBE>
__global__ __launch_bounds__(NTHREADS) void attn_fwd_kernel(Params p) {
  using C = Cfg<DT, D>;
  __shared__ __attribute__((aligned(16))) uint8_t smem[2 * C::BUF];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int i32 = lane & 31;
  const int g = lane >> 5;

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

  // ---- Q block in registers (MFMA B operand: lane holds row i32, k-half g)
  constexpr int NKQ = DT == DT_BF16 ? D / 16 : D / 64;
  const int qload = min(qrow, S - 1);
  const uint8_t* qptr = p.q + (q_head + qload) * C::RB;
  bf16x8 qb16[DT == DT_BF16 ? NKQ : 1];
  i32x8 qf8[DT == DT_FP8 ? NKQ : 1];
  if constexpr (DT == DT_BF16) {
#pragma unroll
    for (int kk = 0; kk < NKQ; ++kk)
      qb16[kk] = *(const bf16x8*)(qptr + (16 * kk + 8 * g) * 2);
  } else {
#pragma unroll
    for (int kk = 0; kk < NKQ; ++kk) {
      const u32x4 lo = *(const u32x4*)(qptr + 64 * kk + 32 * g);
      const u32x4 hi = *(const u32x4*)(qptr + 64 * kk + 32 * g + 16);
      qf8[kk] = i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3],
                      (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
    }
  }

  // ---- staging of one key tile: global -> registers -> LDS
  u32x4 kreg[C::KCH];
  u32x4 vreg[DT == DT_BF16 ? C::VCH : 1];
  u32x2 vreg8[DT == DT_FP8 ? 4 : 1];
  auto load_tile = [&](int t) {
    const int key0 = t * BC;
#pragma unroll
    for (int c = 0; c < C::KCH; ++c) {
      const int cid = tid + c * NTHREADS;
      const int row = cid / C::NCH, ch = cid % C::NCH;
      const int key = min(key0 + row, S - 1);
      kreg[c] = *(const u32x4*)(kg + (size_t)key * C::RB + ch * 16);
      if constexpr (DT == DT_BF16) vreg[c] = *(const u32x4*)(vg + (size_t)key * C::RB + ch * 16);
    }
    if constexpr (DT == DT_FP8) {
      // item (key group of 4, 8-column chunk); D/8 chunks per key row
      constexpr int NDC = D / 8;
      if (tid < (BC / 4) * NDC) {
        const int kgp = tid / NDC, dc = tid % NDC;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int key = min(key0 + 4 * kgp + e, S - 1);
          vreg8[e] = *(const u32x2*)(vg + (size_t)key * C::RB + dc * 8);
        }
      }
    }
  };
  auto store_tile = [&](int buf) {
    uint8_t* kl = smem + buf * C::BUF;
    uint8_t* vl = kl + C::KT;
#pragma unroll
    for (int c = 0; c < C::KCH; ++c) {
      const int cid = tid + c * NTHREADS;
      const int row = cid / C::NCH, ch = cid % C::NCH;
      *(u32x4*)(kl + k_off<DT, D>(row, ch)) = kreg[c];
      if constexpr (DT == DT_BF16) *(u32x4*)(vl + v_off<DT, D>(row, ch * 16)) = vreg[c];
    }
    if constexpr (DT == DT_FP8) {
      constexpr int NDC = D / 8;
      if (tid < (BC / 4) * NDC) {
        const int kgp = tid / NDC, dc = tid % NDC;
        const int pos = vt_pos(4 * kgp);
        // 4 keys x 8 columns of bytes -> 8 columns x 4 keys (byte transpose)
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const uint32_t x0 = vreg8[0][half], x1 = vreg8[1][half];
          const uint32_t x2 = vreg8[2][half], x3 = vreg8[3][half];
          const uint32_t a_lo = __builtin_amdgcn_perm(x1, x0, 0x05010400u);
          const uint32_t a_hi = __builtin_amdgcn_perm(x1, x0, 0x07030602u);
          const uint32_t b_lo = __builtin_amdgcn_perm(x3, x2, 0x05010400u);
          const uint32_t b_hi = __builtin_amdgcn_perm(x3, x2, 0x07030602u);
          const uint32_t col[4] = {__builtin_amdgcn_perm(b_lo, a_lo, 0x05040100u),
                                   __builtin_amdgcn_perm(b_lo, a_lo, 0x07060302u),
                                   __builtin_amdgcn_perm(b_hi, a_hi, 0x05040100u),
                                   __builtin_amdgcn_perm(b_hi, a_hi, 0x07060302u)};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int d = dc * 8 + half * 4 + e;
            *(uint32_t*)(vl + d * C::VPITCH + pos) = col[e];
          }
        }
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

  load_tile(0);
  store_tile(0);
  __syncthreads();

  for (int t = 0; t < ntiles; ++t) {
    const int buf = t & 1;
    if (t + 1 < ntiles) load_tile(t + 1);
    const int kt0 = t * BC;
    const bool active = wave_live && (!CAUSAL || kt0 <= qw0 + WROWS - 1);
    if (active) {
      const uint8_t* kl = smem + buf * C::BUF;
      const uint8_t* vl = kl + C::KT;

      // ---- S^T = K Q^T for the 128 keys of the tile (4 blocks of 32 keys)
      f32x16 sacc[4];
#pragma unroll
      for (int kb = 0; kb < 4; ++kb) sacc[kb] = f32x16{0.0f};
      const int krow = i32;
#pragma unroll
      for (int kk = 0; kk < NKQ; ++kk) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb) {
          const int row = kb * 32 + krow;
          if constexpr (DT == DT_BF16) {
            const bf16x8 a = *(const bf16x8*)(kl + k_off<DT, D>(row, 2 * kk + g));
            sacc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, qb16[kk], sacc[kb], 0, 0, 0);
          } else {
            const u32x4 lo = *(const u32x4*)(kl + k_off<DT, D>(row, 4 * kk + 2 * g));
            const u32x4 hi = *(const u32x4*)(kl + k_off<DT, D>(row, 4 * kk + 2 * g + 1));
            const i32x8 a = i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3],
                                  (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
            sacc[kb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, qf8[kk], sacc[kb], 0, 0,
                                                                       0, 0, 0, 0);
          }
        }
      }
      // accumulator value j of block kb holds key kt0 + 32 kb + 8 (j/4) + 4 g + j%4

      // ---- masking: causal diagonal and the ragged tail only
      const bool need_mask = (CAUSAL && kt0 + BC - 1 > qw0) || (kt0 + BC > S);
      if (need_mask) {
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const int key = kt0 + kb * 32 + 8 * (j >> 2) + 4 * g + (j & 3);
            const bool bad = (CAUSAL && key > qrow) || key >= S;
            if (bad) sacc[kb][j] = -INFINITY;
          }
      }

      const bool probe_row = PROBE && b == p.pb && h == p.ph && qrow >= p.prow0 &&
                             qrow < p.prow0 + p.pnrows;
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

      // ---- running maximum (threshold 0: moves to the maximum so far)
      float mt = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 4; ++kb)
#pragma unroll
        for (int j = 0; j < 16; ++j) mt = __builtin_fmaxf(mt, sacc[kb][j]);
      mt = __builtin_fmaxf(mt, __shfl_xor(mt, 32));
      const float m_new = __builtin_fmaxf(m_run, mt);
      const float alpha = __builtin_amdgcn_exp2f((m_run - m_new) * p.c1);
      m_run = m_new;

      // ---- weights, in place over the scores
      float tsum = 0.0f;
      if constexpr (MODE == MODE_H15) {
        const float nb2 = __builtin_fmaf(-m_new, p.c2, 2.0f * off);
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const float s = sacc[kb][j];
            float w = h15_weight(s, p.c2, nb2);
            if (need_mask && s == -INFINITY) w = 0.0f;
            sacc[kb][j] = w;
            tsum += w;
          }
      } else {
        const float nb1 = __builtin_fmaf(-m_new, p.c1, off);
#pragma unroll
        for (int kb = 0; kb < 4; ++kb)
#pragma unroll
          for (int j = 0; j < 16; ++j) {
            const float w = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc[kb][j], p.c1, nb1));
            sacc[kb][j] = w;
            tsum += w;
          }
      }
      l_part = l_part * alpha + tsum;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int j = 0; j < 16; ++j) oacc[db][j] *= alpha;

      // ---- P in the operand type, then O^T += V^T P^T
      if constexpr (DT == DT_BF16) {
        bf16x8 pb[8];
#pragma unroll
        for (int ks = 0; ks < 8; ++ks)
#pragma unroll
          for (int r = 0; r < 8; ++r) pb[ks][r] = (__bf16)sacc[ks >> 1][8 * (ks & 1) + r];
        if constexpr (PROBE) {
          if (probe_row) {
            const size_t rbase = (size_t)(qrow - p.prow0) * S;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
              for (int j = 0; j < 16; ++j) {
                const int key = kt0 + kb * 32 + 8 * (j >> 2) + 4 * g + (j & 3);
                if (key < S) {
                  const __bf16 pv = pb[2 * kb + (j >> 3)][j & 7];
                  p.w_out[rbase + key] = sacc[kb][j];
                  p.p_out[rbase + key] = (uint32_t)__builtin_bit_cast(uint16_t, pv);
                }
              }
          }
        }
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
#pragma unroll
          for (int ks = 0; ks < 8; ++ks) {
            // keys of this 16-key step: base + 8 (r/4) + 4 g + r%4, r = 0..7
            const int base = 16 * ks;
            const int G4 = lane >> 4, L = lane & 15;
            const int key_a = base + 4 * (G4 >> 1) + (L >> 2);
            const int col = 32 * db + 16 * (G4 & 1) + 4 * (L & 3);
            const bf16x4v lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                (__attribute__((address_space(3))) bf16x4v*)(vl + v_off<DT, D>(key_a, col * 2)));
            const bf16x4v hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                (__attribute__((address_space(3))) bf16x4v*)(vl + v_off<DT, D>(key_a + 8, col * 2)));
            const bf16x8 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
            oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pb[ks], oacc[db], 0, 0, 0);
          }
        }
      } else {
        i32x8 pf[2];
#pragma unroll
        for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
          for (int w4 = 0; w4 < 8; ++w4) {
            const int kb = 2 * t2 + (w4 >> 2), j0 = 4 * (w4 & 3);
            uint32_t word = 0;
            word = __builtin_amdgcn_cvt_pk_fp8_f32(sacc[kb][j0], sacc[kb][j0 + 1], word, false);
            word = __builtin_amdgcn_cvt_pk_fp8_f32(sacc[kb][j0 + 2], sacc[kb][j0 + 3], word, true);
            pf[t2][w4] = (int)word;
          }
        if constexpr (PROBE) {
          if (probe_row) {
            const size_t rbase = (size_t)(qrow - p.prow0) * S;
#pragma unroll
            for (int kb = 0; kb < 4; ++kb)
#pragma unroll
              for (int j = 0; j < 16; ++j) {
                const int key = kt0 + kb * 32 + 8 * (j >> 2) + 4 * g + (j & 3);
                if (key < S) {
                  const uint32_t word = (uint32_t)pf[kb >> 1][4 * (kb & 1) + (j >> 2)];
                  p.w_out[rbase + key] = sacc[kb][j];
                  p.p_out[rbase + key] = (word >> (8 * (j & 3))) & 0xFFu;
                }
              }
          }
        }
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const int d = 32 * db + i32;
#pragma unroll
          for (int t2 = 0; t2 < 2; ++t2) {
            const u32x4 lo = *(const u32x4*)(vl + d * C::VPITCH + (2 * t2) * 32 + 16 * g);
            const u32x4 hi = *(const u32x4*)(vl + d * C::VPITCH + (2 * t2 + 1) * 32 + 16 * g);
            const i32x8 a = i32x8{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3],
                                  (int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
            oacc[db] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, pf[t2], oacc[db], 0, 0,
                                                                       0, 0, 0, 0);
          }
        }
      }
    }
    if (t + 1 < ntiles) store_tile(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue: O = acc / l * v_descale (bf16), LSE
  if (!wave_live) return;
  const float l = l_part + __shfl_xor(l_part, 32);
  if (qrow >= S) return;
  const float inv = p.vd / l;
  uint16_t* orow = p.o + (q_head + qrow) * (size_t)D;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int jq = 0; jq < 4; ++jq) {
      const int col = 32 * db + 8 * jq + 4 * g;
      uint32_t w01, w23;
      {
        const __bf16 a0 = (__bf16)(oacc[db][4 * jq + 0] * inv);
        const __bf16 a1 = (__bf16)(oacc[db][4 * jq + 1] * inv);
        const __bf16 a2 = (__bf16)(oacc[db][4 * jq + 2] * inv);
        const __bf16 a3 = (__bf16)(oacc[db][4 * jq + 3] * inv);
        w01 = (uint32_t)__builtin_bit_cast(uint16_t, a0) | ((uint32_t)__builtin_bit_cast(uint16_t, a1) << 16);
        w23 = (uint32_t)__builtin_bit_cast(uint16_t, a2) | ((uint32_t)__builtin_bit_cast(uint16_t, a3) << 16);
      }
      *(u32x2*)(orow + col) = u32x2{w01, w23};
    }
  if (p.lse && g == 0)
    p.lse[q_head + qrow] = 0.69314718055994531f * (m_run * p.c1 + log2f(l) - off);
}

// Probe support: pre-fill the probe buffers (s = -inf, w = 0, P = 0).
__global__ void probe_fill(float* s, float* w, uint32_t* pbits, size_t n) {
  const size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    s[i] = -INFINITY;
    w[i] = 0.0f;
    pbits[i] = 0u;
  }
}

template <int DT, int D, bool CAUSAL, int MODE, bool PROBE>
hipError_t launch_one(const Params& p, hipStream_t st) {
  const unsigned grid = (unsigned)(p.nqb * p.B * p.Hq);
  hipLaunchKernelGGL((attn_fwd_kernel<DT, D, CAUSAL, MODE, PROBE>), dim3(grid), dim3(NTHREADS), 0,
                     st, p);
  return hipGetLastError();
}

template <int DT, int D, bool PROBE>
hipError_t launch_dt_d(const Params& p, int causal, int mode, hipStream_t st) {
  if (causal) {
    return mode == ATTN_EXP_H15 ? launch_one<DT, D, true, MODE_H15, PROBE>(p, st)
                                : launch_one<DT, D, true, MODE_EXACT, PROBE>(p, st);
  }
  return mode == ATTN_EXP_H15 ? launch_one<DT, D, false, MODE_H15, PROBE>(p, st)
                              : launch_one<DT, D, false, MODE_EXACT, PROBE>(p, st);
}

template <bool PROBE>
hipError_t launch_any(const Params& p, int dtype, int d, int causal, int mode, hipStream_t st) {
  if (dtype == ATTN_BF16)
    return d == 128 ? launch_dt_d<DT_BF16, 128, PROBE>(p, causal, mode, st)
                    : launch_dt_d<DT_BF16, 64, PROBE>(p, causal, mode, st);
  return d == 128 ? launch_dt_d<DT_FP8, 128, PROBE>(p, causal, mode, st)
                  : launch_dt_d<DT_FP8, 64, PROBE>(p, causal, mode, st);
}

bool finite_pos(float x) { return x > 0.0f && x < INFINITY; }

int fill_params(Params& p, const void* q, const void* k, const void* v, void* o, float* lse, int B,
                int Hq, int Hkv, int S, int d, int causal, float scale, int dtype, int exp_mode,
                const attn_opts* opts) {
  (void)causal;
  if (!q || !k || !v || !o) return ATTN_EINVAL;
  if (B <= 0 || Hq <= 0 || Hkv <= 0 || S <= 0 || d <= 0) return ATTN_EINVAL;
  if (Hq % Hkv != 0) return ATTN_EINVAL;
  if (!finite_pos(scale)) return ATTN_EINVAL;
  if (dtype != ATTN_BF16 && dtype != ATTN_FP8_E4M3) return ATTN_EUNSUPPORTED;
  if (exp_mode != ATTN_EXP_EXACT && exp_mode != ATTN_EXP_H15) return ATTN_EUNSUPPORTED;
  if (d != 64 && d != 128) return ATTN_EUNSUPPORTED;
  const uintptr_t mis = (uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)o;
  if (mis & 15u) return ATTN_EUNSUPPORTED;
  if (lse && ((uintptr_t)lse & 3u)) return ATTN_EUNSUPPORTED;
  float qd = 1.0f, kd = 1.0f, vd = 1.0f;
  if (dtype == ATTN_FP8_E4M3) {
    if (!opts) return ATTN_EINVAL;
    qd = opts->q_descale;
    kd = opts->k_descale;
    vd = opts->v_descale;
    if (!finite_pos(qd) || !finite_pos(kd) || !finite_pos(vd)) return ATTN_EINVAL;
  }
  const long long rows = (long long)B * Hq * S;
  if (rows > (1LL << 31) / 2) return ATTN_EUNSUPPORTED;
  p = Params{};
  p.q = (const uint8_t*)q;
  p.k = (const uint8_t*)k;
  p.v = (const uint8_t*)v;
  p.o = (uint16_t*)o;
  p.lse = lse;
  p.B = B;
  p.Hq = Hq;
  p.Hkv = Hkv;
  p.S = S;
  p.G = Hq / Hkv;
  // base-two exponent scale of a raw logit; the H15 path uses the doubled
  // constant (App. B.1), the rescale factor and LSE the plain one
  p.c1 = (float)((double)scale * (double)qd * (double)kd * 1.4426950408889634);
  p.c2 = 2.0f * p.c1;
  p.vd = vd;
  p.nqb = (S + BR - 1) / BR;
  p.remap = ((B * Hkv) % 8 == 0) ? 1 : 0;
  return ATTN_OK;
}

}  // namespace

extern "C" {

int attn_tile_bc(void) { return BC; }

const char* attn_strerror(int code) {
  switch (code) {
    case ATTN_OK: return "ok";
    case ATTN_EINVAL: return "invalid argument";
    case ATTN_EUNSUPPORTED: return "unsupported configuration";
    case ATTN_ELAUNCH: return "kernel launch failed";
    default: return "unknown error code";
  }
}

int attn_fwd_ex(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
                int Hkv, int S, int d, int causal, float scale, int dtype, int exp_mode,
                const attn_opts* opts) {
  Params p;
  const int rc = fill_params(p, q, k, v, o, lse, B, Hq, Hkv, S, d, causal, scale, dtype, exp_mode, opts);
  if (rc != ATTN_OK) return rc;
  hipStream_t st = opts ? (hipStream_t)opts->stream : nullptr;
  const hipError_t e = launch_any<false>(p, dtype, d, causal ? 1 : 0, exp_mode, st);
  return e == hipSuccess ? ATTN_OK : ATTN_ELAUNCH;
}

int attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
             int Hkv, int S, int d, int causal, float scale, int dtype, int exp_mode) {
  return attn_fwd_ex(q, k, v, o, lse, B, Hq, Hkv, S, d, causal, scale, dtype, exp_mode, nullptr);
}

int attn_fwd_probe(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
                   int Hkv, int S, int d, int causal, float scale, int dtype, int exp_mode,
                   const attn_opts* opts, int b, int h, int row0, int nrows, float* s_out,
                   float* w_out, uint32_t* p_bits_out) {
  Params p;
  const int rc = fill_params(p, q, k, v, o, lse, B, Hq, Hkv, S, d, causal, scale, dtype, exp_mode, opts);
  if (rc != ATTN_OK) return rc;
  if (!s_out || !w_out || !p_bits_out) return ATTN_EINVAL;
  if (b < 0 || b >= B || h < 0 || h >= Hq || row0 < 0 || nrows < 1 || row0 + nrows > S)
    return ATTN_EINVAL;
  p.pb = b;
  p.ph = h;
  p.prow0 = row0;
  p.pnrows = nrows;
  p.s_out = s_out;
  p.w_out = w_out;
  p.p_out = p_bits_out;
  hipStream_t st = opts ? (hipStream_t)opts->stream : nullptr;
  const size_t n = (size_t)nrows * (size_t)S;
  hipLaunchKernelGGL(probe_fill, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, s_out, w_out,
                     p_bits_out, n);
  if (hipGetLastError() != hipSuccess) return ATTN_ELAUNCH;
  hipError_t e;
  e = launch_any<true>(p, dtype, d, causal ? 1 : 0, exp_mode, st);
  return e == hipSuccess ? ATTN_OK : ATTN_ELAUNCH;
}

}  // extern "C"
