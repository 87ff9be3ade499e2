// The C entry points declared in h15attn.h: argument checks, the per-call
// constants of the method (the base-two logit scale c1 and its 2^k multiple,
// App. B.1 "Implementation"; the offset of the FP8 weights), the choice of
// kernel variant, the decode cut into key parts and its workspace, then the
// launchers of h15attn.hip.  Plain C++: no HIP types or calls here, so the
// same checks build with a host compiler alone under the sanitizers.
#include <math.h>
#include <stddef.h>
#include <stdint.h>

#include "attn_params.h"
#include "h15attn.h"

using namespace h15;

namespace {

bool finite_pos(float x) { return x > 0.0f && x < INFINITY; }

// Input-rounding order k of an ABI exp_mode (0 for the exact control).
int exp_order(int exp_mode) {
  switch (exp_mode) {
    case ATTN_EXP_H15: return 1;
    case ATTN_EXP_SQ4: return 2;
    case ATTN_EXP_SQ8: return 3;
    default: return 0;
  }
}

// Kernel variant for an ABI exp_mode.  For FP8 every raw logit satisfies
// |s| <= d * 448^2, so |y| <= 2 ck d 448^2 + 8 * 2^k with ck = 2^k c1; when
// that is below 2^15 the rounded integer n = RNE(y) fits an int16 lane and
// the clamp can be taken there (the narrow mode).
int kernel_mode(int dtype, int exp_mode, int d, float ck) {
  if (exp_mode == ATTN_EXP_ROWMAX_POT) return MODE_ROWMAX_POT;
  const int k = exp_order(exp_mode);
  if (k == 0) return MODE_EXACT;
  if (dtype == ATTN_FP8_E4M3) {
    const double ymax = 2.0 * (double)ck * (double)d * 448.0 * 448.0 * (1.0 + 1e-5) + 8.0 * (1 << k);
    if (ymax < 32767.0) return 2 * k;
  }
  return 2 * k - 1;
}

// The compact layout (4-wave groups, two per CU) for BF16 grids where a
// group's prologue, barriers and epilogue are poorly hidden: short rows
// (S <= 2048: few key tiles per group) or fewer default groups (8 waves,
// 256 query rows) than two per compute unit.  Measured on MI355X (H15 and
// the exact control alike): +4% at causal B4 Hq32 S2K, +11..27% at causal
// 1K-4K with 16 heads; at 8K with 16 heads and at 16K with 64 heads the
// default layout is level or ahead for the control, so it stays there.
constexpr int COMPACT_MAX_S = 2048;
constexpr long long COMPACT_BELOW_GROUPS = 512;

// 1 when the forward call takes the compact layout: BF16 (FP8 groups are 4
// waves already) and any weight but Rowmax-PoT (whose first pass
// double-buffers K).
int use_compact(int dtype, int exp_mode, int B, int Hq, int S) {
  if (dtype != ATTN_BF16 || exp_mode == ATTN_EXP_ROWMAX_POT) return 0;
  const long long groups = (long long)B * Hq * ((S + FWD_ROWS_BF16 - 1) / FWD_ROWS_BF16);
  return (S <= COMPACT_MAX_S || groups < COMPACT_BELOW_GROUPS) ? 1 : 0;
}

// query rows per workgroup for an operand type and layout
int row_block(int dtype, int compact) {
  if (compact) return FWD_ROWS_COMPACT;
  return dtype == ATTN_FP8_E4M3 ? FWD_ROWS_FP8 : FWD_ROWS_BF16;
}

int fill_params(Params& p, const void* q, const void* k, const void* v, void* o, float* lse, int B,
                int Hq, int Hkv, int S, int d, float scale, int dtype, int exp_mode,
                const attn_opts* opts) {
  if (!q || !k || !v || !o) return ATTN_EINVAL;
  if (B <= 0 || Hq <= 0 || Hkv <= 0 || S <= 0 || d <= 0) return ATTN_EINVAL;
  if (Hq % Hkv != 0) return ATTN_EINVAL;
  if (!finite_pos(scale)) return ATTN_EINVAL;
  if (dtype != ATTN_BF16 && dtype != ATTN_FP8_E4M3) return ATTN_EUNSUPPORTED;
  if (exp_mode != ATTN_EXP_EXACT && exp_mode != ATTN_EXP_ROWMAX_POT && exp_order(exp_mode) == 0)
    return ATTN_EUNSUPPORTED;
  // Rowmax-PoT: 21 levels 2^0 .. 2^-20 need bf16's range for P (e4m3 spans
  // under 18 octaves); its anchor is the whole-row maximum, so no threshold
  if (exp_mode == ATTN_EXP_ROWMAX_POT && (dtype != ATTN_BF16 || (opts && opts->rescale_threshold != 0.0f)))
    return ATTN_EUNSUPPORTED;
  if (d != 64 && d != 128) return ATTN_EUNSUPPORTED;
  const uintptr_t mis = (uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)o;
  if (mis & 15u) return ATTN_EUNSUPPORTED;
  if (lse && ((uintptr_t)lse & 3u)) return ATTN_EUNSUPPORTED;
  float qd = 1.0f, kd = 1.0f, vd = 1.0f;
  const float tau = opts ? opts->rescale_threshold : 0.0f;
  if (!(tau >= 0.0f && tau <= 64.0f)) return ATTN_EINVAL;
  if (dtype == ATTN_FP8_E4M3) {
    if (!opts) return ATTN_EINVAL;
    if (tau != 0.0f) return ATTN_EUNSUPPORTED;
    qd = opts->q_descale;
    kd = opts->k_descale;
    vd = opts->v_descale;
    if (!finite_pos(qd) || !finite_pos(kd) || !finite_pos(vd)) return ATTN_EINVAL;
  }
  const long long rows = (long long)B * Hq * S;
  if (rows > (1LL << 31) / 2) return ATTN_EUNSUPPORTED;
  // one head's K or V rows are addressed with 32-bit byte offsets
  if ((long long)S * d * (dtype == ATTN_BF16 ? 2 : 1) > INT32_MAX) return ATTN_EUNSUPPORTED;
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
  // base-two exponent scale of a raw logit; the weight uses 2^k times it
  // (the doubled constant of App. B.1 for k = 1; the scaling is exact), the
  // rescale factor and LSE the plain one
  p.c1 = (float)((double)scale * (double)qd * (double)kd * 1.4426950408889634);
  p.ck = ldexpf(p.c1, exp_order(exp_mode));
  p.vd = vd;
  p.tau = tau;
  p.tau_wave = (opts && opts->rescale_per_wave) ? 1 : 0;
  p.compact = use_compact(dtype, exp_mode, B, Hq, S);
  p.nqb = (S + row_block(dtype, p.compact) - 1) / row_block(dtype, p.compact);
  p.remap = ((B * Hkv) % 8 == 0) ? 1 : 0;
  return ATTN_OK;
}


// Number of key parts for a cut of split_keys keys (0 or >= Sk: one part).
int dec_parts(int Sk, int split_keys) {
  if (split_keys <= 0 || split_keys >= Sk) return 1;
  return (Sk + split_keys - 1) / split_keys;
}

size_t dec_workspace_bytes(long long rows, int nsplit, int d) {
  if (nsplit <= 1) return 0;
  return (size_t)rows * (size_t)nsplit * ((size_t)d + 2) * sizeof(float);
}

int fill_dec_params(DecParams& p, const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
                    int Hkv, int Sq, int Sk, int Sk_cap, int d, float scale, int dtype, int exp_mode,
                    int split_keys, const attn_opts* opts) {
  if (!q || !k || !v || !o) return ATTN_EINVAL;
  if (B <= 0 || Hq <= 0 || Hkv <= 0 || Sq <= 0 || Sk <= 0 || Sk_cap <= 0 || d <= 0) return ATTN_EINVAL;
  if (Hq % Hkv != 0 || Sq > Sk || Sk > Sk_cap) return ATTN_EINVAL;
  if (!finite_pos(scale)) return ATTN_EINVAL;
  if (split_keys < 0 || split_keys % BC != 0) return ATTN_EINVAL;
  if (dtype != ATTN_BF16 && dtype != ATTN_FP8_E4M3) return ATTN_EUNSUPPORTED;
  if (exp_mode != ATTN_EXP_EXACT && exp_order(exp_mode) == 0) return ATTN_EUNSUPPORTED;
  if (d != 64 && d != 128) return ATTN_EUNSUPPORTED;
  const uintptr_t mis = (uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)o;
  if (mis & 15u) return ATTN_EUNSUPPORTED;
  if (lse && ((uintptr_t)lse & 3u)) return ATTN_EUNSUPPORTED;
  float qd = 1.0f, kd = 1.0f, vd = 1.0f;
  if (opts && !(opts->rescale_threshold == 0.0f)) {
    // the parts take the running maximum as their anchor: threshold 0 only
    return (opts->rescale_threshold >= 0.0f && opts->rescale_threshold <= 64.0f) ? ATTN_EUNSUPPORTED
                                                                                  : ATTN_EINVAL;
  }
  if (dtype == ATTN_FP8_E4M3) {
    if (!opts) return ATTN_EINVAL;
    qd = opts->q_descale;
    kd = opts->k_descale;
    vd = opts->v_descale;
    if (!finite_pos(qd) || !finite_pos(kd) || !finite_pos(vd)) return ATTN_EINVAL;
  }
  const long long rows = (long long)B * Hq * Sq;
  if (rows > (1LL << 30)) return ATTN_EUNSUPPORTED;
  // one head's cache is addressed with 32-bit byte offsets
  if ((long long)Sk_cap * d * (dtype == ATTN_BF16 ? 2 : 1) > INT32_MAX) return ATTN_EUNSUPPORTED;
  const int G = Hq / Hkv;
  const long long R = (long long)G * Sq;
  const long long nrb = (R + DEC_ROWS - 1) / DEC_ROWS;
  const int nsplit = dec_parts(Sk, split_keys);
  if ((long long)B * Hkv * nrb * nsplit > INT32_MAX) return ATTN_EUNSUPPORTED;
  p = DecParams{};
  p.q = (const uint8_t*)q;
  p.k = (const uint8_t*)k;
  p.v = (const uint8_t*)v;
  p.o = (uint16_t*)o;
  p.lse = lse;
  p.B = B;
  p.Hq = Hq;
  p.Hkv = Hkv;
  p.Sq = Sq;
  p.Sk = Sk;
  p.Sk_cap = Sk_cap;
  p.G = G;
  p.R = (int)R;
  p.nrb = (int)nrb;
  p.nsplit = nsplit;
  p.split_keys = nsplit == 1 ? ((Sk + BC - 1) / BC) * BC : split_keys;
  p.c1 = (float)((double)scale * (double)qd * (double)kd * 1.4426950408889634);
  p.ck = ldexpf(p.c1, exp_order(exp_mode));
  p.vd = vd;
  return ATTN_OK;
}

// Points the parts' partial results into the workspace (several parts only).
int bind_workspace(DecParams& p, int d, void* workspace, size_t workspace_bytes) {
  if (p.nsplit > 1) {
    const size_t need = dec_workspace_bytes((long long)p.B * p.Hq * p.Sq, p.nsplit, d);
    if (!workspace || ((uintptr_t)workspace & 15u) || workspace_bytes < need) return ATTN_EINVAL;
    p.part_o = (float*)workspace;
    p.part_ml = (float*)workspace + (size_t)p.B * p.Hq * p.Sq * p.nsplit * d;
  }
  return ATTN_OK;
}

int decode_launch(const DecParams& p, int dtype, int d, int causal, int exp_mode, void* st, bool probe) {
  const int mode = kernel_mode(dtype, exp_mode, d, p.ck);
  return launch_decode(p, dtype, d, causal, mode, st, probe) == 0 ? ATTN_OK : ATTN_ELAUNCH;
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
    case ATTN_ENOSPACE: return "the decode cut needs more workspace than the built-in scratch buffer";
    default: return "unknown error code";
  }
}

int attn_fwd_ex(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
                int Hkv, int S, int d, int causal, float scale, int dtype, int exp_mode,
                const attn_opts* opts) {
  Params p;
  const int rc = fill_params(p, q, k, v, o, lse, B, Hq, Hkv, S, d, scale, dtype, exp_mode, opts);
  if (rc != ATTN_OK) return rc;
  if (p.remap && !causal) p.remap = 2;
  void* st = opts ? opts->stream : nullptr;
  const int mode = kernel_mode(dtype, exp_mode, d, p.ck);
  return launch_fwd(p, dtype, d, causal ? 1 : 0, mode, st, false) == 0 ? ATTN_OK : ATTN_ELAUNCH;
}

int attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
             int Hkv, int S, int d, int causal, float scale, int dtype, int exp_mode) {
  // unit descales (FP8 values are taken as stored), default stream, threshold 0
  const attn_opts unit = {1.0f, 1.0f, 1.0f, nullptr, 0.0f, 0};
  return attn_fwd_ex(q, k, v, o, lse, B, Hq, Hkv, S, d, causal, scale, dtype, exp_mode, &unit);
}

int attn_fwd_probe(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
                   int Hkv, int S, int d, int causal, float scale, int dtype, int exp_mode,
                   const attn_opts* opts, int b, int h, int row0, int nrows, float* s_out,
                   float* w_out, uint32_t* p_bits_out) {
  Params p;
  const int rc = fill_params(p, q, k, v, o, lse, B, Hq, Hkv, S, d, scale, dtype, exp_mode, opts);
  if (rc != ATTN_OK) return rc;
  if (p.remap && !causal) p.remap = 2;
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
  void* st = opts ? opts->stream : nullptr;
  const size_t n = (size_t)nrows * (size_t)S;
  if (launch_probe_fill(s_out, w_out, p_bits_out, n, st) != 0) return ATTN_ELAUNCH;
  const int mode = kernel_mode(dtype, exp_mode, d, p.ck);
  return launch_fwd(p, dtype, d, causal ? 1 : 0, mode, st, true) == 0 ? ATTN_OK : ATTN_ELAUNCH;
}

int attn_decode_split_keys(int B, int Hq, int Hkv, int Sq, int Sk, int d, int dtype) {
  (void)d;
  (void)dtype;
  if (B <= 0 || Hq <= 0 || Hkv <= 0 || Sq <= 0 || Sk <= 0 || Hq % Hkv != 0) return 0;
  // aim at two workgroups per compute unit (512), with at least eight tiles
  // of keys per part (measured on MI355X at 4K-32K caches: parts of four
  // tiles ran 10-25% slower than parts of eight, whose copies have time to
  // stream behind the first ones)
  const long long nrb = ((long long)(Hq / Hkv) * Sq + DEC_ROWS - 1) / DEC_ROWS;
  const long long groups = (long long)B * Hkv * nrb;
  const long long tiles = (Sk + BC - 1) / BC;
  long long parts = (512 + groups - 1) / groups;
  if (parts > tiles / 8) parts = tiles / 8;
  if (parts <= 1) return 0;
  const long long per = (tiles + parts - 1) / parts;
  return (int)(per * BC);
}

size_t attn_decode_workspace_bytes(int B, int Hq, int Sq, int Sk, int d, int split_keys) {
  if (B <= 0 || Hq <= 0 || Sq <= 0 || Sk <= 0 || d <= 0 || split_keys < 0) return 0;
  return dec_workspace_bytes((long long)B * Hq * Sq, dec_parts(Sk, split_keys), d);
}

int attn_decode(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq, int Hkv,
                int Sq, int Sk, int Sk_cap, int d, int causal, float scale, int dtype, int exp_mode,
                int split_keys, void* workspace, size_t workspace_bytes, const attn_opts* opts) {
  DecParams p;
  const int rc = fill_dec_params(p, q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, Sk_cap, d, scale, dtype, exp_mode,
                                 split_keys, opts);
  if (rc != ATTN_OK) return rc;
  const int wrc = bind_workspace(p, d, workspace, workspace_bytes);
  if (wrc != ATTN_OK) return wrc;
  void* st = opts ? opts->stream : nullptr;
  return decode_launch(p, dtype, d, causal ? 1 : 0, exp_mode, st, false);
}

int attn_decode_noalloc(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq, int Hkv,
                        int Sq, int Sk, int Sk_cap, int d, int causal, float scale, int dtype, int exp_mode,
                        int split_keys, const attn_opts* opts) {
  DecParams p;
  const int rc = fill_dec_params(p, q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, Sk_cap, d, scale, dtype, exp_mode,
                                 split_keys, opts);
  if (rc != ATTN_OK) return rc;
  // the parts' partial results go to the built-in workspace of the current
  // device (nothing is allocated); a cut that needs more is refused
  const size_t need = dec_workspace_bytes((long long)B * Hq * Sq, p.nsplit, d);
  if (need > scratch_capacity()) return ATTN_ENOSPACE;
  void* st = opts ? opts->stream : nullptr;
  void* ws = nullptr;
  if (need > 0) {
    const int src = scratch_address(st, &ws);
    if (src == 2) return ATTN_EINVAL;
    if (src != 0) return ATTN_ELAUNCH;
  }
  const int wrc = bind_workspace(p, d, ws, need);
  if (wrc != ATTN_OK) return wrc;
  return decode_launch(p, dtype, d, causal ? 1 : 0, exp_mode, st, false);
}

int attn_decode_probe(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq, int Hkv,
                      int Sq, int Sk, int Sk_cap, int d, int causal, float scale, int dtype, int exp_mode,
                      int split_keys, void* workspace, size_t workspace_bytes, const attn_opts* opts, int b,
                      int h, int i, float* s_out, float* w_out, uint32_t* p_bits_out) {
  DecParams p;
  const int rc = fill_dec_params(p, q, k, v, o, lse, B, Hq, Hkv, Sq, Sk, Sk_cap, d, scale, dtype, exp_mode,
                                 split_keys, opts);
  if (rc != ATTN_OK) return rc;
  if (!s_out || !w_out || !p_bits_out) return ATTN_EINVAL;
  if (b < 0 || b >= B || h < 0 || h >= Hq || i < 0 || i >= Sq) return ATTN_EINVAL;
  const int wrc = bind_workspace(p, d, workspace, workspace_bytes);
  if (wrc != ATTN_OK) return wrc;
  p.pb = b;
  p.ph = h;
  p.pi = i;
  p.s_out = s_out;
  p.w_out = w_out;
  p.p_out = p_bits_out;
  void* st = opts ? opts->stream : nullptr;
  const size_t n = (size_t)Sk;
  if (launch_probe_fill(s_out, w_out, p_bits_out, n, st) != 0) return ATTN_ELAUNCH;
  return decode_launch(p, dtype, d, causal ? 1 : 0, exp_mode, st, true);
}

}  // extern "C"
