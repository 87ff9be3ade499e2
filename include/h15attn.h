/*
 * h15attn: fused attention forward for AMD Instinct MI355X (gfx950) whose
 * softmax exponential is either the hardware exp2 (the control) or
 * Rowmax-H15, from "Approximating Softmax in Pretrained LLMs: Model
 * Sensitivity and Kernel Acceleration".
 *
 * Operation (App. A.1, Eq. (exact-attention), with the valid key set V(i) =
 * {j : j <= i} when causal, else every key):
 *     O[b,h,i,:] = sum_{j in V(i)} p_ij V[b,h/G,j,:],   G = Hq / Hkv,
 *     p_ij = w_ij / sum_{j in V(i)} w_ij,
 * computed online over key tiles of attn_tile_bc() keys with a running row
 * maximum m (FlashAttention-style).  The weight w_ij is
 *   ATTN_EXP_EXACT: exp2(c1 * (s_ij - m) + off), hardware exp2;
 *   ATTN_EXP_H15:   Rowmax-H15 of the base-two exponent x = c1*(s_ij - m)
 *                   + off (Sec. 5.2 Eq. (m-h15); App. B.1 "Implementation"):
 *                   n = RNE(2x), w = (1 + (n mod 2)/2) * 2^floor(n/2),
 *                   realised as y = fma(s, c2, fma(-m, c2, 2 off)),
 *                   y = max(y, -252), t = y + 0x1.8p23f (RNE),
 *                   w = bits^-1((bits(t) << 22) + bits(1.0f)), c2 = 2*c1.
 *   ATTN_EXP_SQ4, ATTN_EXP_SQ8: the finer input rounding S(Q_{2^-k}(x)) for
 *                   k = 2 and k = 3 (App. B.2 "Exponential-map ablation";
 *                   Rowmax-H15 is k = 1): Q_{2^-k}(x) = 2^-k RNE(2^k x),
 *                   S(q) = 2^floor(q) (1 + q - floor(q)) (App. B.1), realised
 *                   as the H15 sequence, the input scaled by 2^k, not 2:
 *                   y = fma(s, ck, fma(-m, ck, 2^k off)), ck = 2^k c1,
 *                   y = max(y, -126 * 2^k), t = y + 0x1.8p23f (RNE),
 *                   w = bits^-1((bits(t) << (23 - k)) + bits(1.0f)).
 *                   Every weight has at most k mantissa bits, so P = w is
 *                   exact in bf16, and in e4m3 from 2^-6 up.
 *   ATTN_EXP_ROWMAX_POT: Rowmax-PoT (App. A.6 Eq. (rowmax-pot)), anchored at
 *                   the whole-row maximum m of the raw logits (a first pass
 *                   over the key tiles computes it, so the running maximum
 *                   never moves): x = fp32(fp32(m - s_ij) * c1),
 *                   d = min(20, floor(x + 1/2)), w = 2^-d.  BF16 only (the 21
 *                   levels are exact in bf16; e4m3 spans under 18 octaves).
 * where s_ij = sum_c q_ic k_jc is the raw logit of the stored operands (bf16
 * values, or e4m3 values without their descales) accumulated in fp32,
 * c1 = fp32(scale * q_descale * k_descale * log2(e)) (products in double,
 * in that order), off = 0 for BF16 and 8 for FP8 (so P = w <= 2^8 fits
 * e4m3), and m the running maximum of the raw logits, moved at every key
 * tile to the maximum so far (rescale threshold 0, App. B.2: per-tile
 * running max).  The row sum and the PV product consume the same weights:
 * l sums w in fp32; PV multiplies V by P = w stored as bf16 (exact for the
 * approximate weights)
 * or e4m3 (round to nearest even).  Output:
 *     O = (sum_j P_j V_j) / l * v_descale, stored as bf16;
 *     LSE = ln2 * (m * c1 + log2(l) - off)   (natural log of the normaliser
 *           of the scaled logits; for H15 the approximated normaliser).
 *
 * Layouts: every tensor is contiguous BHSD (batch, head, sequence, head
 * dim).  q: [B][Hq][S][d]; k, v: [B][Hkv][S][d]; o: [B][Hq][S][d] bf16;
 * lse: [B][Hq][S] fp32 (may be NULL).  Elements are bf16 (2 bytes) or OCP
 * e4m3fn (1 byte) according to dtype.  Query head h reads key/value head
 * h / (Hq / Hkv).  Causal masking is top-left aligned (query i sees keys
 * j <= i).
 *
 * Memory and streams: all pointers are device pointers owned by the caller;
 * the library allocates, frees and synchronises nothing.  Calls are
 * asynchronous on the given stream (NULL: the default stream); buffers must
 * stay valid until the stream reaches the work.  The library holds no state
 * and may be called from several threads, except for the built-in decode
 * workspace of attn_decode_noalloc (one buffer per GPU, shared by its calls).
 *
 * Errors: arguments are validated before anything is launched; on error
 * nothing is written.  Every entry point returns ATTN_OK or a negative code,
 * described by attn_strerror().
 */
#ifndef H15ATTN_H
#define H15ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum attn_dtype { ATTN_BF16 = 0, ATTN_FP8_E4M3 = 1 };
enum attn_expmode {
    ATTN_EXP_EXACT = 0,
    ATTN_EXP_H15 = 1,
    ATTN_EXP_SQ4 = 2,
    ATTN_EXP_SQ8 = 3,
    ATTN_EXP_ROWMAX_POT = 4 /* BF16 only, rescale_threshold 0 (else ATTN_EUNSUPPORTED) */
};
enum attn_status {
    ATTN_OK = 0,
    ATTN_EINVAL = -1,      /* null pointer, non-positive size, Hq % Hkv != 0,
                              scale or descale not positive and finite,
                              rescale_threshold outside [0, 64] */
    ATTN_EUNSUPPORTED = -2, /* d not in {64, 128}, unknown dtype or exp_mode,
                              pointer not 16-byte aligned, B*Hq*S > 2^30, or
                              one head's K/V rows (S * d * element bytes)
                              not addressable with 31-bit offsets */
    ATTN_ELAUNCH = -3,     /* the HIP runtime reported an error (a launch, or
                              naming the device for attn_decode_noalloc) */
    ATTN_ENOSPACE = -4     /* attn_decode_noalloc: the cut needs more workspace
                              than the built-in buffer holds */
};

/* Optional per-call settings.  FP8 requires the three per-tensor descales
 * (the factors that turn stored e4m3 values back into real values); BF16
 * ignores them.  stream is a hipStream_t (NULL: default stream).
 *
 * rescale_threshold (tau, base-two units, default 0) is the conditional
 * rescale of App. B.2 ("Conditional rescaling moves the anchor"): at each key
 * tile the running maximum m moves to max(m, mt) only when it grows by more
 * than tau, g = fp32(fp32(mt - m) * c1) > tau (the first tile always sets
 * it); otherwise the anchor stays and the weights of the tile are taken
 * relative to it (they may exceed 2^off, up to about 2^(tau + off)).  With
 * rescale_per_wave = 0 each row decides for itself (the paper's semantic
 * simulation); with 1 the decision is shared by each aligned group of 32
 * query rows (rows 32w .. 32w + 31 of a head), moving every row's anchor when
 * any real row of the group grows by more than tau (FlashAttention-4's
 * per-warp decision).  tau must be finite, 0 <= tau <= 64 (else
 * ATTN_EINVAL); FP8 requires tau = 0 (P must stay within e4m3's range; else
 * ATTN_EUNSUPPORTED).  A zero-initialised struct gives tau = 0. */
typedef struct attn_opts {
    float q_descale, k_descale, v_descale;
    void* stream;
    float rescale_threshold;
    int rescale_per_wave;
} attn_opts;

/* Attention forward on the default stream with unit descales (FP8 operands
 * are taken at their stored e4m3 values) and rescale threshold 0: the same as
 * attn_fwd_ex with opts = {1, 1, 1, NULL, 0, 0}. */
int attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
             int Hkv, int S, int d, int causal, float scale, int dtype, int exp_mode);

/* Attention forward with descales and a stream (opts may be NULL for BF16). */
int attn_fwd_ex(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
                int Hkv, int S, int d, int causal, float scale, int dtype, int exp_mode,
                const attn_opts* opts);

/* Test access to the method's intermediate values.  Runs the same kernel code
 * as attn_fwd_ex (same tiles, same arithmetic, O and LSE written identically)
 * and, for query rows [row0, row0 + nrows) of head (b, h), also stores the
 * fp32 raw logits s, the fp32 weights w and the stored P bits (bf16 pattern
 * or e4m3 code, zero-extended) of every key: s_out, w_out, p_bits_out are
 * device buffers of nrows * S elements, row-major.  Entries of masked keys
 * are written as s = -inf, w = 0, P = 0.  The weight stored is the one
 * computed at the key's tile, relative to the running maximum of that time
 * (before later rescales).  Requires 0 <= row0, nrows >= 1,
 * row0 + nrows <= S, 0 <= b < B, 0 <= h < Hq; otherwise ATTN_EINVAL. */
int attn_fwd_probe(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
                   int Hkv, int S, int d, int causal, float scale, int dtype, int exp_mode,
                   const attn_opts* opts, int b, int h, int row0, int nrows, float* s_out,
                   float* w_out, uint32_t* p_bits_out);

/* ---- Decode over a key/value cache -------------------------------------
 *
 * Sq query rows per query head attend to the first Sk rows of a key/value
 * cache (App. A.1's attention with the queries of the last Sq positions; the
 * paper leaves decode outside its scope, this is the library's extension).
 * Query position i (0 <= i < Sq) sees keys j <= Sk - Sq + i when causal
 * (bottom-right alignment: the last query row sees the whole cache; with
 * Sq = Sk it is attn_fwd's causal mask), every key otherwise.
 *
 * Key parts: the keys are cut into consecutive parts of split_keys keys (a
 * multiple of attn_tile_bc(); 0, or any value >= Sk, gives one part), which
 * run in parallel.  Within a part the weights follow the recurrence described
 * above for attn_fwd, over the part's keys only: its tiles start at the
 * part's first key and its running maximum starts afresh, so for the lattice
 * weights (ATTN_EXP_H15, SQ4, SQ8) the cut is part of the result (each
 * weight is rounded relative to its own part's running maximum).  The parts
 * then merge exactly:
 *     m = max_p m_p,   f_p = 2^(c1 (m_p - m)),   l = sum_p f_p l_p,
 *     O = (sum_p f_p O_p) / l * v_descale,   LSE = ln2 (m c1 + log2 l - off),
 * with m_p, l_p, O_p a part's final running maximum, row sum and unnormalised
 * output (parts holding no visible key of a row take no part in its merge).
 * With one part the result equals attn_fwd's rows of the same keys.  The
 * exact control does not depend on the cut beyond rounding.  For a given
 * split_keys the result is deterministic; attn_decode_split_keys() proposes
 * one that fills the GPU and is a function of the shape only.
 *
 * Layouts: q: [B][Hq][Sq][d]; k, v: [B][Hkv][Sk_cap][d], the first Sk rows of
 * each head being the cache (rows Sk .. Sk_cap - 1 are never read); o:
 * [B][Hq][Sq][d] bf16; lse: [B][Hq][Sq] fp32 (may be NULL).  Element types,
 * GQA mapping, descales, stream and exp_mode as for attn_fwd_ex; the rescale
 * threshold must be 0 and Rowmax-PoT is not offered (ATTN_EUNSUPPORTED).
 *
 * Workspace: with more than one part the library keeps each part's (m, l, O)
 * in a caller-provided device buffer of at least
 * attn_decode_workspace_bytes() bytes, 16-byte aligned (else ATTN_EINVAL);
 * with one part it may be NULL.  Nothing in it needs initialising; two calls
 * in flight at once must not share it.  The call launches two kernels on the
 * stream (the parts, then their merge), one when there is a single part.
 *
 * Errors (besides those of attn_fwd_ex): ATTN_EINVAL for Sq > Sk,
 * Sk > Sk_cap, split_keys negative or not a multiple of attn_tile_bc(), or a
 * missing or short workspace; ATTN_EUNSUPPORTED for one head's cache of
 * Sk_cap * d * element bytes beyond 2^31 - 1, B * Hq * Sq > 2^30, or a
 * nonzero rescale threshold. */
int attn_decode(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq, int Hkv,
                int Sq, int Sk, int Sk_cap, int d, int causal, float scale, int dtype, int exp_mode,
                int split_keys, void* workspace, size_t workspace_bytes, const attn_opts* opts);

/* Bytes of workspace attn_decode needs for this shape and cut (0 for one
 * part, or for invalid sizes). */
size_t attn_decode_workspace_bytes(int B, int Hq, int Sq, int Sk, int d, int split_keys);

/* A cut (split_keys) for attn_decode that gives about two workgroups per
 * compute unit with at least eight key tiles per part, or 0 (one part) when
 * the shape fills the GPU without cutting.  A function of its arguments
 * only; 0 for invalid sizes. */
int attn_decode_split_keys(int B, int Hq, int Hkv, int Sq, int Sk, int d, int dtype);

/* attn_decode for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid allocation):
 * the same kernels and results as attn_decode with the same split_keys, but
 * the parts' partial results go to a workspace built into the library, one
 * 16 MiB buffer per GPU (allocated when the library's code is loaded on that
 * GPU and held until the process ends), instead of a caller's buffer.  The
 * call allocates and frees nothing.  Every call on one GPU shares that GPU's
 * buffer: calls that may overlap on one GPU (other streams, other threads)
 * race and give wrong results; calls in stream order are safe.  Nothing in
 * the buffer needs clearing (every part writes all of its partial results
 * before the merge reads them).  The first call on a device looks up that
 * device's buffer with the device current.
 *
 * The buffer used is the current device's, so a stream passed in opts must
 * belong to the current device.
 *
 * Errors: those of attn_decode (without the workspace ones); ATTN_ENOSPACE
 * when attn_decode_workspace_bytes() of the shape and cut exceeds 16 MiB
 * (16777216 bytes; choose a coarser cut, or use attn_decode); ATTN_EINVAL
 * when the stream belongs to another device; nothing is launched then. */
int attn_decode_noalloc(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq, int Hkv,
                        int Sq, int Sk, int Sk_cap, int d, int causal, float scale, int dtype, int exp_mode,
                        int split_keys, const attn_opts* opts);

/* Test access to decode's intermediate values, as attn_fwd_probe: runs the
 * same kernels as attn_decode (O and LSE written identically) and stores, for
 * query row (b, h, i), the fp32 raw logits s, the fp32 weights w (relative
 * to the running maximum of the key's tile within its part) and the P bits
 * of every cache key: s_out, w_out, p_bits_out are device buffers of Sk
 * elements.  Keys the row does not see are written as s = -inf, w = 0,
 * P = 0.  Requires 0 <= b < B, 0 <= h < Hq, 0 <= i < Sq (else ATTN_EINVAL). */
int attn_decode_probe(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq, int Hkv,
                      int Sq, int Sk, int Sk_cap, int d, int causal, float scale, int dtype, int exp_mode,
                      int split_keys, void* workspace, size_t workspace_bytes, const attn_opts* opts, int b,
                      int h, int i, float* s_out, float* w_out, uint32_t* p_bits_out);

/* Static description of an error code. */
const char* attn_strerror(int code);

/* Key-tile width of the online recurrence (the running maximum moves once per
 * tile of this many keys, in increasing key order). */
int attn_tile_bc(void);

#ifdef __cplusplus
}
#endif

#endif /* H15ATTN_H */
