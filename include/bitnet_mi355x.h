/*
 * bitnet_mi355x.h -- C ABI of the ternary-weight x int8-activation mpGEMM library for AMD MI355X (gfx950).
 *
 * The library computes the mixed-precision GEMM/GEMV that Bitnet.cpp (arXiv 2502.11880) identifies as the
 * bulk of ternary-LLM inference time (abstract; Sec. 1), in three calls that follow the phases of the
 * paper's algorithms (Algorithm "MAD-based mpGEMM", Algorithm "ELUT mpGEMM", Algorithms TL1/TL2):
 *
 *   bitnet_pack_weights   offline weight preprocessing: absmean ternarisation + packing (Sec. 2.1, Table 1)
 *   bitnet_quantize_act   per-call activation preprocessing: per-token absmax int8 (Sec. 2.1, Sec. 3.2.2)
 *   bitnet_mpgemm         accumulation + dequantisation: y[m, n] = beta / s_m * sum_k xq[m, k] * t[n, k]
 *
 * Conventions shared by every entry point
 *   - Every tensor pointer is a DEVICE pointer (hipMalloc or equivalent) to contiguous row-major memory
 *     owned by the caller.  The library never allocates, frees or copies between host and device.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).  All work is enqueued on it;
 *     no call synchronises.  Results are ready when the stream reaches them.
 *   - Arguments are validated on the host before anything is enqueued; a non-OK status means nothing was
 *     enqueued (except BITNET_E_HIP, which reports a failed launch).  No call aborts or throws.
 *   - Calls are thread-safe.  Two calls that run concurrently must not share a workspace.
 *   - Naming: M = tokens (activation rows), N = output features (weight rows), K = reduction length.
 */
#ifndef BITNET_MI355X_H
#define BITNET_MI355X_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    BITNET_OK = 0,
    BITNET_E_INVALID = 1,    /* null pointer, unknown option, or a buffer smaller than required      */
    BITNET_E_SHAPE = 2,      /* a size outside the supported range (see each call)                   */
    BITNET_E_ALIGN = 3,      /* a device pointer not aligned to 16 bytes                             */
    BITNET_E_LAYOUT = 4,     /* unknown weight layout                                                */
    BITNET_E_WORKSPACE = 5,  /* workspace missing or smaller than the matching *_workspace_bytes     */
    BITNET_E_HIP = 6         /* the HIP runtime reported an error; see bitnet_last_error()          */
} bitnet_status;

/*
 * Weight layouts.  All need N % 16 == 0 and K % 64 == 0 (rows are tiled by 16, K by 64).
 *
 * BITNET_LAYOUT_I2S ("Int2 with a Scale", Table 1, Sec. 3.2.2): 2 bits per weight, code = t + 1.
 *   16-row groups; K in blocks of up to 256 (four 64-k sub-tiles; only the last block may be shorter).
 *   In a block of T sub-tiles the group's 64 lanes l = 16*q + r (r = row in group, q = 0..3) own 4*T
 *   contiguous bytes each; word j of lane (r, q) holds k = 64*(4*s + j) + 16*q + 4*f + b in byte b,
 *   bits [2f, 2f+1].  Size N*K/4 bytes.
 *
 * BITNET_LAYOUT_TL2 (Sec. 3.1, Table 5, Table 6): ~1.67 bits per weight.  K splits into
 *   ThreeK = floor(K/384)*384 and TwoK = K - ThreeK (block-fitting weight splitting, Sec. 3.1.2).
 *   Each triple of the ThreeK part becomes a 4-bit index |9 t0 + 3 t1 + t2| and a 1-bit sign [value < 0]
 *   (Table 6, mirror consolidation Sec. 3.1.1), stored in separate planes (signed-unsigned weight
 *   splitting, Sec. 3.1.2); each pair of the TwoK part becomes the 4-bit TL1 code 3(t0+1) + (t1+1)
 *   (Table 5).  Planes in order: index [N*ThreeK/6 B], sign [N*ThreeK/24 B], tail [N*TwoK/4 B].
 *   In a 384-k block, lane l = 16*q + r owns 16 index bytes (triples 32q..32q+31 of the block, triple i
 *   in byte i/2, low nibble first) and 4 sign bytes (triple i at bit i%8 of byte i/8).  The tail is cut
 *   into 64-k units; lane (r, q) owns one 32-bit word per unit holding pairs 32u + 8q + i (byte i/2, low
 *   nibble first), with each lane's words contiguous.
 *
 * BITNET_LAYOUT_TL1 (Table 1 "TL1_1", Algorithm TL1, Table 5): 2 bits per weight.  Every pair of weights is its
 *   4-bit Table 5 code 3(t0+1) + (t1+1), in the tiling of I2_S: a 32-bit word of lane (r, q) in sub-tile j of
 *   block s holds the 16 weights k = 64*(4*s + j) + 16*q + e of row 16R + r as 8 pair codes, pair i (weights
 *   e = 2i, 2i+1) in byte i % 4, low nibble for i < 4 and high nibble for i >= 4.  Size N*K/4 bytes.
 *
 * Integer-weight layouts (Appendix "Insight", Table 3, Algorithm "ELUT mpGEMM"): weights from a set of C consecutive
 * integers, packed from int8 values with bitnet_pack_int_weights and multiplied by table lookups (Eq. 3, with the
 * sign operation of Eq. 5 where the set is symmetric).  Row-major planes; group j of row n is weights g j .. g j+g-1.
 * BITNET_LAYOUT_C4G2: C = 4 {-2, -1, 0, 1}, g = 2, code 4 (w0 + 2) + (w1 + 2) in 4 bits (group j in byte
 *   n K/4 + j/2, low nibble first); 2 bits per weight.  Size N*K/4.
 * BITNET_LAYOUT_C5G2: C = 5 {-2, .., 2}, g = 2, 4-bit index |5 w0 + w1| placed as C4G2's codes, then a sign plane
 *   of one bit per group (group j of row n at byte N K/4 + n K/16 + j/8, bit j % 8); 2.5 bits per weight.
 *   Size N*K/4 + N*K/16.
 * BITNET_LAYOUT_C3G5: C = 3 {-1, 0, 1}, g = 5, one byte per group at n K/5 + j: index |sum_i 3^(4-i) w_i| (0..121)
 *   in bits 0-6, sign [sum < 0] in bit 7; 1.6 bits per weight.  Needs K % 320 == 0.  Size N*K/5.
 *
 * Lossy kernels (Table 1 "TL2_0", "TL1_0"; Sec. 3.2.1): BITNET_LAYOUT_TL2_0 and BITNET_LAYOUT_TL1_0 pack exactly as
 *   TL2 and TL1, but bitnet_mpgemm looks the groups up in tables quantised to int8: per token and table block (the
 *   128 triples of a 384-k TL2 block, or the 32 pairs of a 64-k TL1 unit) every entry is divided by 2^s, s the
 *   smallest shift that brings the block's largest |entry| within 127, and rounded half to even; the block's sum
 *   is multiplied back by 2^s.  The accumulators are exact integers of that rule, close to but not equal to
 *   sum_k xq t (the paper's lossy kernels; the quantisation itself is this library's reading).
 */
typedef enum {
    BITNET_LAYOUT_I2S = 0,
    BITNET_LAYOUT_TL2 = 1,
    BITNET_LAYOUT_TL1 = 2,
    BITNET_LAYOUT_C4G2 = 3,
    BITNET_LAYOUT_C5G2 = 4,
    BITNET_LAYOUT_C3G5 = 5,
    BITNET_LAYOUT_TL2_0 = 6,
    BITNET_LAYOUT_TL1_0 = 7
} bitnet_layout;

/* Bytes of the packed buffer for an N x K weight in `layout`; 0 if the shape or layout is unsupported. */
size_t bitnet_packed_bytes(int layout, int64_t N, int64_t K);

/* Workspace bytes bitnet_pack_weights needs for an N x K weight (independent of the layout). */
size_t bitnet_pack_workspace_bytes(int64_t N, int64_t K);

/*
 * bitnet_pack_weights -- ternarise and pack one weight tensor (Sec. 2.1; Algorithm TL1/TL2 weight
 * preprocessing; Table 1 for I2_S).
 *   W          device fp32 [N, K], finite values.
 *   packed     device buffer of at least bitnet_packed_bytes(layout, N, K) bytes; fully overwritten.
 *   w_scale    device fp32 [1]; receives beta = the fp32 value nearest (ties to even) to the exact mean
 *              of |W| over all N*K entries, so it does not depend on any summation order.
 *   t = clamp(rint(fp32(W / beta)), -1, 1) with IEEE division and ties-to-even; beta == 0 gives t = 0.
 *   ws         device workspace of bitnet_pack_workspace_bytes(N, K) bytes (any contents).
 *   Shapes: N % 16 == 0, K % 64 == 0, N*K < 2^32.  Pointers 16-byte aligned.
 */
bitnet_status bitnet_pack_weights(int layout, const float* W, int64_t N, int64_t K,
                                  void* packed, size_t packed_bytes, float* w_scale,
                                  void* ws, size_t ws_bytes, void* stream);

/*
 * bitnet_pack_int_weights -- pack integer weights for an integer-weight layout (C4G2, C5G2, C3G5; Table 3).
 *   Wq         device int8 [N, K], values in the layout's set (a value outside it is packed as the nearest value
 *              of the set).  The per-tensor scale is the caller's: pass it to bitnet_mpgemm as w_scale.
 *   packed     device buffer of at least bitnet_packed_bytes(layout, N, K) bytes; fully overwritten.
 *   Shapes: N % 16 == 0, K % 64 == 0 (C3G5: K % 320 == 0), N*K < 2^32.  Pointers 16-byte aligned.
 */
bitnet_status bitnet_pack_int_weights(int layout, const int8_t* Wq, int64_t N, int64_t K, void* packed,
                                      size_t packed_bytes, void* stream);

/*
 * bitnet_quantize_act -- per-token absmax int8 quantisation (Sec. 2.1, Sec. 3.2.2).
 *   x         device fp32 [M, K], finite values.
 *   xq        device int8 [M, K]:  xq = clamp(rint(fp32(x * s_m)), -128, 127)  (ties to even).
 *   x_scale   device fp32 [M]:     s_m = fp32(127 / max(max_k |x[m, k]|, 1e-5)).
 *   x_rowsum  device int32 [M] or NULL: sum_k xq[m, k].  Passing it on to bitnet_mpgemm saves the I2_S
 *             kernels the work of forming it (their codes are t + 1, so they subtract this sum).
 *   Shapes: M >= 1, 1 <= K <= 1048576.  x and xq 16-byte aligned, x_scale and x_rowsum 4-byte.
 */
bitnet_status bitnet_quantize_act(const float* x, int64_t M, int64_t K, int8_t* xq, float* x_scale,
                                  int32_t* x_rowsum, void* stream);

/* Workspace bytes bitnet_mpgemm needs for this problem (0 is a valid answer). */
size_t bitnet_mpgemm_workspace_bytes(int layout, int64_t M, int64_t N, int64_t K);

/*
 * bitnet_mpgemm -- ternary x int8 accumulation with the dequantisation epilogue (Eq. 1 / Eq. 3).
 *   packed, packed_bytes, w_scale   as written by bitnet_pack_weights for an N x K weight in `layout`.
 *   xq, x_scale                     as written by bitnet_quantize_act for an M x K activation.
 *   x_rowsum                        as written by bitnet_quantize_act, or NULL (then computed here).
 *   y      device fp32 [M, N]: y[m, n] = fp32(acc[m, n]) * fp32(w_scale / x_scale[m]).
 *   acc    device int32 [M, N] or NULL: when given, also receives acc[m, n] = sum_k xq[m, k] * t[n, k]
 *          exactly (the same integers for every tiling and launch shape).  A parity output: with it the
 *          prefill and multi-token kernels run an instance that also stores the sums, a few percent slower.
 *   ws     device workspace of at least bitnet_mpgemm_workspace_bytes(layout, M, N, K) bytes, or NULL when
 *          that is 0 (else BITNET_E_WORKSPACE).  It holds the exact int32 partial sums of a prefill GEMM split
 *          along K (M > 16, small grids; only when x_rowsum is given) and, for TL2 with M > 16, the weights
 *          rewritten in the I2_S layout (N * K / 4 bytes) that the prefill GEMM reads; any contents on entry,
 *          nothing kept between calls.  Calls that run concurrently must not share it.
 *   Shapes: M >= 1, N % 16 == 0, K % 64 == 0, K <= 132096 (127 * K < 2^24 keeps acc exact in fp32);
 *   I2_S and TL1 also need N * K and M * K below 2^32.  I2_S: M <= 16 runs the decode GEMV; 17 <= M <= 112 with
 *   x_rowsum given and K <= 16384 runs the same GEMV in slices of up to 16 tokens, one launch for all slices (the
 *   small-batch regime between decode and prefill, which the paper leaves open, Sec. "Limitations"); larger M the
 *   prefill GEMM.  TL1: the same decode GEMV (the pair codes expanded to int8 in registers) where I2_S runs it;
 *   otherwise the weights are rewritten in the I2_S layout in the workspace (N * K / 4 bytes) for the prefill GEMM.
 *   Integer-weight layouts (C4G2, C5G2, C3G5): table lookups with the tables built in LDS for 4 tokens at a time
 *   (2 for C3G5), any M; x_rowsum is not used and no workspace is needed.  TL2_0 and TL1_0: the lossy table
 *   lookups described with the layouts, 8 tokens per launch, any M, no workspace; acc receives their integers.
 *   TL2: one token runs the table lookups of Eq. 3 (tables built in LDS) where the row's tables fit (K <= 14336);
 *   otherwise, up to 16 tokens with 384 <= K < 18816, the packed triples are expanded to int8 weights and
 *   multiplied on int8 MFMA; more than 16 tokens (with N * K and M * K below 2^32) rewrite the weights in the
 *   I2_S layout in the workspace and run the I2_S prefill GEMM; the remaining shapes run the table lookups in
 *   slices of 8 tokens.
 */
bitnet_status bitnet_mpgemm(int layout, const void* packed, size_t packed_bytes, const float* w_scale,
                            int64_t N, int64_t K, const int8_t* xq, const float* x_scale,
                            const int32_t* x_rowsum, int64_t M, float* y, int32_t* acc, void* ws,
                            size_t ws_bytes, void* stream);

/*
 * bitnet_mpgemm_noalloc -- bitnet_mpgemm without a workspace argument, for callers that cannot allocate device
 * memory: code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc.
 *   Arguments, results, shapes and statuses as bitnet_mpgemm.  The workspace bitnet_mpgemm would take (split-K
 *   slices of the prefill GEMM, TL2 weights rewritten for it) comes from a static device array of
 *   BITNET_NOALLOC_SCRATCH_BYTES (32 MiB) that each GPU the library runs on holds until the process ends.  A shape
 *   whose bitnet_mpgemm_workspace_bytes exceeds it returns BITNET_E_WORKSPACE before anything is enqueued.
 *   Every call on one GPU shares that GPU's array and leaves its contents behind (nothing in it has to start at
 *   zero): calls on one stream are ordered, but calls that overlap on one GPU (other streams, other threads) race.
 *   The call allocates and frees nothing; on its first use on a device it looks the array's address up once.
 */
#define BITNET_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
bitnet_status bitnet_mpgemm_noalloc(int layout, const void* packed, size_t packed_bytes, const float* w_scale,
                                    int64_t N, int64_t K, const int8_t* xq, const float* x_scale,
                                    const int32_t* x_rowsum, int64_t M, float* y, int32_t* acc, void* stream);

/*
 * Workspace bytes with which bitnet_mpgemm_fused runs every split it can use for these n_linears weights (host
 * array N of rows, shared K, M tokens; 0 is a valid answer and 0 is also returned for invalid arguments): at
 * least the largest bitnet_mpgemm_workspace_bytes of the weights (the minimum the call accepts), and for a fused
 * I2_S prefill launch (M > 16), which splits K over all its weights at once, enough for that split.  Given less
 * (but at least that minimum), the fused launch runs without splitting.
 */
size_t bitnet_mpgemm_fused_workspace_bytes(int layout, int n_linears, const int64_t* N, int64_t K, int64_t M);

/*
 * bitnet_mpgemm_fused -- one activation, several weights: bitnet_quantize_act followed by bitnet_mpgemm for
 * each weight, as one launch where possible (the linears that read the same input, such as q/k/v or gate/up).
 * Results are identical to those separate calls.
 *   n_linears                   1..8.
 *   packed, packed_bytes, w_scale, N, y
 *                               HOST arrays of n_linears entries: device packed buffer, its size, device beta,
 *                               rows of that weight, device fp32 output [M, N[i]].
 *   K, x, M                     the shared reduction length and the device fp32 activation [M, K]; x may be
 *                               NULL when xq, x_scale and x_rowsum already hold its quantised form (as written
 *                               by bitnet_quantize_act): then they are inputs and only the products run.
 *   xq, x_scale, x_rowsum       device outputs as in bitnet_quantize_act (all three required).
 *   ws                          as for bitnet_mpgemm, at least the largest workspace of the n products
 *                               (bitnet_mpgemm_fused_workspace_bytes lets a prefill launch split K).
 *   Shapes: 1 <= M <= 2^24; each weight as in bitnet_mpgemm.  I2_S with M == 1 and K <= 61440 runs as one
 *   launch (every work group quantises the row itself, keeping the codes in LDS); other I2_S cases run the
 *   quantiser and then all products in one launch (the decode GEMV for M <= 16, the prefill GEMM over the
 *   weights' concatenated row tiles above).  TL2 with M == 1 and 384 <= K < 18816 also runs as one launch (the
 *   row quantised in every work group, the triples expanded for MFMA); other TL2 cases run the quantiser and
 *   then one launch for all weights (the MFMA expansion for M <= 16 and K < 18816; for M > 16, every weight
 *   rewritten in the I2_S layout and one prefill launch, where ws holds all of them) or one bitnet_mpgemm call
 *   per weight.  TL1 runs as I2_S up to 16 tokens (the same launches, the pair codes expanded in registers) and
 *   as TL2 above (every weight rewritten in the I2_S layout, one prefill launch).  The integer-weight layouts run
 *   the quantiser and then the table lookups of each weight.
 */
bitnet_status bitnet_mpgemm_fused(int layout, int n_linears, const void* const* packed, const size_t* packed_bytes,
                                  const float* const* w_scale, const int64_t* N, int64_t K, const float* x,
                                  int64_t M, int8_t* xq, float* x_scale, int32_t* x_rowsum, float* const* y,
                                  void* ws, size_t ws_bytes, void* stream);

/*
 * bitnet_elut_tables -- the activation tables of the TL2 path, written out (Eq. 3; mirror consolidation,
 * Sec. 3.1.1; the Table-setup step of Algorithm "ELUT mpGEMM" and PreCompute of Algorithms TL1/TL2).
 * bitnet_mpgemm builds the same tables in LDS for the TL2 layout; this call exposes them.
 *   xq    device int8 [M, K] (from bitnet_quantize_act).
 *   lut   device int16 [M, ThreeK/3, 16]: for triple g (k = 3g..3g+2) entry i < 14 is
 *         d0(i)*xq[3g] + d1(i)*xq[3g+1] + d2(i)*xq[3g+2] where i = 9*d0 + 3*d1 + d2 with digits in {-1,0,1}
 *         and a non-negative leading digit; entries 14 and 15 are 0.
 *   lut1  device int16 [M, TwoK/2, 16]: for tail pair p (k = ThreeK + 2p, +1) entry i < 9 is
 *         (i/3 - 1)*xq[k] + (i%3 - 1)*xq[k+1] (Table 5 order); entries 9..15 are 0.  May be NULL when TwoK == 0.
 *   Shapes: K % 64 == 0, 384 <= K <= 132096, ThreeK = floor(K/384)*384, TwoK = K - ThreeK.
 */
bitnet_status bitnet_elut_tables(const int8_t* xq, int64_t M, int64_t K, int16_t* lut, int16_t* lut1,
                                 void* stream);

/* Static description of a status code. */
const char* bitnet_status_string(int status);

/* Detail text of the last non-OK status returned on the calling thread ("" if none). */
const char* bitnet_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* BITNET_MI355X_H */
