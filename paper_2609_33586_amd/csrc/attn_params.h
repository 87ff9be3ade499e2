// Host-side interface between the C entry points (attn_api.cpp: argument
// checks and the per-call constants, plain C++) and the gfx950 kernels
// (h15attn.hip: kernels and their launchers).  Nothing here depends on HIP,
// so the argument checks also build with a host compiler alone (the
// sanitizer build of the checks).
#ifndef H15ATTN_PARAMS_H
#define H15ATTN_PARAMS_H

#include <stddef.h>
#include <stdint.h>

namespace h15 {

constexpr int WROWS = 32;  // query rows per wave
constexpr int BC = 128;    // keys per tile (the running max moves once per tile)
// query rows per forward workgroup: 4 waves for FP8, 8 for BF16
constexpr int FWD_ROWS_FP8 = 4 * WROWS;
constexpr int FWD_ROWS_BF16 = 8 * WROWS;
// the compact layout (BF16 grids that underfill the chip): 4 waves per group
constexpr int FWD_ROWS_COMPACT = 4 * WROWS;
// query rows per decode workgroup
constexpr int DEC_ROWS = WROWS;

// Kernel weight modes.  0 is the exact-exp2 control.  The input-rounding
// family S(Q_{2^-k}) (App. B.2; k = 1 is Rowmax-H15, App. B.1) takes mode
// 2k - 1 with the clamp in FP32 and 2k with the clamp on the rounded integer
// in 16-bit lanes (exact only when |y| < 2^15 for every score).  Mode 7 is
// Rowmax-PoT (App. A.6 Eq. (rowmax-pot)), anchored at the whole-row maximum,
// BF16 only.
enum { MODE_EXACT = 0, MODE_H15 = 1, MODE_H15_NARROW = 2, MODE_ROWMAX_POT = 7 };

// Forward launch parameters.
struct Params {
  const uint8_t* q;
  const uint8_t* k;
  const uint8_t* v;
  uint16_t* o;
  float* lse;
  int B, Hq, Hkv, S, G;
  float c1, ck, vd;  // base-two logit scale; 2^k c1 for the weight; V descale
  float tau;          // conditional-rescale threshold (0: the anchor is the running max)
  int tau_wave;       // 1: the anchor decision is shared by the wave's 32 rows
  int nqb;    // query blocks per head
  int remap;  // XCD-grouped workgroup order: 0 none, 1 query blocks outermost, 2 KV heads outermost
  int compact;  // 1: the compact layout (4-wave groups, at most 80 KB of LDS; BF16 only)
  // probe target (probe launches only)
  int pb, ph, prow0, pnrows;
  float* s_out;
  float* w_out;
  uint32_t* p_out;
};

// Decode launch parameters.
struct DecParams {
  const uint8_t* q;
  const uint8_t* k;
  const uint8_t* v;
  uint16_t* o;
  float* lse;
  float* part_o;   // [rows][nsplit][d], unnormalised O of each part (nsplit > 1)
  float* part_ml;  // [rows][nsplit][2], (m, l) of each part (nsplit > 1)
  int B, Hq, Hkv, Sq, Sk, Sk_cap, G, R, nrb, nsplit, split_keys;
  float c1, ck, vd;
  // probe target (probe launches only): output row (pb, ph, pi)
  int pb, ph, pi;
  float* s_out;
  float* w_out;
  uint32_t* p_out;
};

// Launchers (h15attn.hip).  Each enqueues its kernels on stream (a
// hipStream_t; NULL: the default stream) and returns 0, or nonzero when the
// runtime reports a launch error.  The caller has checked every argument.
int launch_fwd(const Params& p, int dtype, int d, int causal, int mode, void* stream, bool probe);
// the probe buffers pre-filled with s = -inf, w = 0, P = 0 (n elements each)
int launch_probe_fill(float* s, float* w, uint32_t* pbits, size_t n, void* stream);
// the parts' kernel, then (several parts) their merge
int launch_decode(const DecParams& p, int dtype, int d, int causal, int mode, void* stream, bool probe);

// The library's built-in decode workspace (h15attn.hip): its size in bytes,
// and the address of the current device's copy for work on stream (NULL:
// the default stream).  Returns 0; 1 when the runtime cannot name the
// device, the stream's device or the address; 2 when the stream belongs to
// another device than the current one.  The address is looked up once per
// device, on the first call with that device current.
size_t scratch_capacity();
int scratch_address(void* stream, void** ptr);

}  // namespace h15

#endif  // H15ATTN_PARAMS_H
