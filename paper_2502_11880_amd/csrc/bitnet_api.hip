// C ABI of the library: argument validation, layout arithmetic and dispatch to the HIP kernels.
// Every check runs on the host before anything is enqueued; no entry point allocates, frees, copies
// between host and device or synchronises.
#include "bitnet_mi355x.h"
#include "bitnet_internal.hpp"

#include <cstdarg>
#include <cstdio>
#include <mutex>

namespace {

thread_local char g_last_error[512] = "";

bitnet_status fail(bitnet_status st, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_last_error, sizeof(g_last_error), fmt, ap);
    va_end(ap);
    return st;
}

bitnet_status ok() {
    g_last_error[0] = '\0';
    return BITNET_OK;
}

bitnet_status hip_status(hipError_t e, const char* what) {
    if (e == hipSuccess) return ok();
    return fail(BITNET_E_HIP, "%s: %s", what, hipGetErrorString(e));
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

constexpr int64_t kMaxK = 132096;          // 127 * K < 2^24: accumulators stay exact in fp32
constexpr int64_t kDecodeMaxTokens = 16;   // up to 16 tokens fill the rows of one 16x16x64 MFMA

bool weight_shape_ok(int64_t N, int64_t K) {
    return N > 0 && K > 0 && N % bitnet::kRowsPerGroup == 0 && K % bitnet::kSubK == 0 && K <= kMaxK &&
           N <= (int64_t)1 << 30;
}

// c3g5 groups five weights: its rows are whole 64-byte runs of groups (K % 320 == 0)
bool layout_shape_ok(int layout, int64_t N, int64_t K) {
    return weight_shape_ok(N, K) && (layout != BITNET_LAYOUT_C3G5 || K % 320 == 0);
}

bool layout_ok(int layout) {
    return layout >= BITNET_LAYOUT_I2S && layout <= BITNET_LAYOUT_TL1_0;
}

// The lossy kernels (TL2_0, TL1_0) read the packed formats of TL2 and TL1.
bool lossy_layout(int layout) { return layout == BITNET_LAYOUT_TL2_0 || layout == BITNET_LAYOUT_TL1_0; }
int packed_as(int layout) {
    return layout == BITNET_LAYOUT_TL2_0 ? BITNET_LAYOUT_TL2 : layout == BITNET_LAYOUT_TL1_0 ? BITNET_LAYOUT_TL1 : layout;
}

// The integer-weight ELUT layouts (packed from integer weights by bitnet_pack_int_weights)
bool elut_layout(int layout) {
    return layout == BITNET_LAYOUT_C4G2 || layout == BITNET_LAYOUT_C5G2 || layout == BITNET_LAYOUT_C3G5;
}
int elut_format(int layout) {
    return layout == BITNET_LAYOUT_C4G2 ? bitnet::kElutC4G2
           : layout == BITNET_LAYOUT_C5G2 ? bitnet::kElutC5G2 : bitnet::kElutC3G5;
}

// I2_S and TL1 share the tiling, the decode kernels (which read the word format as a template) and their limits.
bool i2s_tiled(int layout) { return layout == BITNET_LAYOUT_I2S || layout == BITNET_LAYOUT_TL1; }
int word_format(int layout) { return layout == BITNET_LAYOUT_TL1 ? bitnet::kFmtTl1 : bitnet::kFmtI2s; }

size_t packed_bytes_of(int layout, int64_t N, int64_t K) {
    layout = packed_as(layout);
    if (i2s_tiled(layout) || layout == BITNET_LAYOUT_C4G2) return (size_t)N * (size_t)K / 4;
    if (layout == BITNET_LAYOUT_C5G2) return (size_t)N * (size_t)K / 4 + (size_t)N * (size_t)K / 16;
    if (layout == BITNET_LAYOUT_C3G5) return (size_t)N * (size_t)K / 5;
    const int64_t three = (K / bitnet::kTl2BlockK) * bitnet::kTl2BlockK;
    const int64_t two = K - three;
    return (size_t)N * three / 6 + (size_t)N * three / 24 + (size_t)N * two / 4;
}

bitnet::FusedLinears one_linear(const void* packed, const float* w_scale, int64_t N, float* y, int32_t* acc) {
    bitnet::FusedLinears L{};
    L.count = 1;
    L.packed[0] = static_cast<const uint8_t*>(packed);
    L.w_scale[0] = w_scale;
    L.y[0] = y;
    L.acc[0] = acc;
    L.N[0] = (int)N;
    bitnet::seal_fused(L);
    return L;
}

// The table lookups of TL2, TL1 (lossy or not) for M tokens of already quantised activations: launches of up to 8
// tokens, each over every weight of L (outputs of later slices offset by the slice's first token).
hipError_t lookup_sliced(bool tl1, bool lossy, const bitnet::FusedLinears& L, const int8_t* xq, const float* x_scale,
                         int64_t M, int64_t K, hipStream_t s) {
    for (int64_t m0 = 0; m0 < M; m0 += bitnet::kElutMaxTokens) {
        const int mc = (int)((M - m0) < bitnet::kElutMaxTokens ? (M - m0) : bitnet::kElutMaxTokens);
        bitnet::FusedLinears Ls = L;
        for (int i = 0; i < L.count; ++i) {
            Ls.y[i] = L.y[i] + m0 * L.N[i];
            Ls.acc[i] = L.acc[i] ? L.acc[i] + m0 * L.N[i] : nullptr;
        }
        const hipError_t e =
            tl1 ? bitnet::launch_tl1_elut_decode(Ls, nullptr, xq + m0 * K, x_scale + m0, mc, (int)K, nullptr, nullptr,
                                                 nullptr, s, lossy)
                : bitnet::launch_tl2_elut_decode(Ls, nullptr, xq + m0 * K, x_scale + m0, mc, (int)K, nullptr, nullptr,
                                                 nullptr, s, lossy);
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}

// TL2 and TL1 at M > 16 run the I2_S prefill GEMM on their weights rewritten in the I2_S layout (in the workspace),
// where the I2_S limits hold.
bool tl2_via_i2s(int64_t M, int64_t N, int64_t K) {
    return M > kDecodeMaxTokens && (uint64_t)N * (uint64_t)K < ((uint64_t)1 << 32) &&
           (uint64_t)M * (uint64_t)K < ((uint64_t)1 << 32);
}

size_t align256(size_t b) { return (b + 255) & ~(size_t)255; }

}  // namespace

extern "C" {

size_t bitnet_packed_bytes(int layout, int64_t N, int64_t K) {
    if (!layout_ok(layout) || !layout_shape_ok(layout, N, K)) return 0;
    return packed_bytes_of(layout, N, K);
}

size_t bitnet_pack_workspace_bytes(int64_t N, int64_t K) {
    (void)N;
    (void)K;
    return bitnet::pack_workspace_bytes();
}

bitnet_status bitnet_pack_weights(int layout, const float* W, int64_t N, int64_t K, void* packed,
                                  size_t packed_bytes, float* w_scale, void* ws, size_t ws_bytes, void* stream) {
    if (!layout_ok(layout)) return fail(BITNET_E_LAYOUT, "unknown layout %d", layout);
    if (elut_layout(layout))
        return fail(BITNET_E_LAYOUT, "layout %d holds integer weights: pack it with bitnet_pack_int_weights", layout);
    if (!W || !packed || !w_scale) return fail(BITNET_E_INVALID, "null pointer argument");
    if (!weight_shape_ok(N, K)) return fail(BITNET_E_SHAPE, "need N %% 16 == 0, K %% 64 == 0, 0 < K <= %lld; got N=%lld K=%lld",
                                            (long long)kMaxK, (long long)N, (long long)K);
    if ((uint64_t)N * (uint64_t)K >= ((uint64_t)1 << 32)) return fail(BITNET_E_SHAPE, "N*K must be below 2^32");
    if (!aligned(W, 16) || !aligned(packed, 16) || !aligned(ws, 16) || !aligned(w_scale, 4))
        return fail(BITNET_E_ALIGN, "W, packed and ws need 16-byte alignment, w_scale 4-byte");
    if (packed_bytes < packed_bytes_of(layout, N, K))
        return fail(BITNET_E_INVALID, "packed buffer holds %zu bytes, %zu needed", packed_bytes,
                    packed_bytes_of(layout, N, K));
    if (!ws || ws_bytes < bitnet::pack_workspace_bytes())
        return fail(BITNET_E_WORKSPACE, "pack workspace needs %zu bytes", bitnet::pack_workspace_bytes());
    return hip_status(bitnet::launch_pack(packed_as(layout), W, N, K, packed, w_scale, ws, (hipStream_t)stream),
                      "bitnet_pack_weights launch");
}

bitnet_status bitnet_pack_int_weights(int layout, const int8_t* Wq, int64_t N, int64_t K, void* packed,
                                      size_t packed_bytes, void* stream) {
    if (!elut_layout(layout)) return fail(BITNET_E_LAYOUT, "layout %d is not an integer-weight ELUT layout", layout);
    if (!Wq || !packed) return fail(BITNET_E_INVALID, "null pointer argument");
    if (!layout_shape_ok(layout, N, K) || (uint64_t)N * (uint64_t)K >= ((uint64_t)1 << 32))
        return fail(BITNET_E_SHAPE, "need N %% 16 == 0, K %% %d == 0, 0 < K <= %lld, N*K < 2^32; got N=%lld K=%lld",
                    layout == BITNET_LAYOUT_C3G5 ? 320 : 64, (long long)kMaxK, (long long)N, (long long)K);
    if (!aligned(Wq, 16) || !aligned(packed, 16)) return fail(BITNET_E_ALIGN, "Wq and packed need 16-byte alignment");
    if (packed_bytes < packed_bytes_of(layout, N, K))
        return fail(BITNET_E_INVALID, "packed buffer holds %zu bytes, %zu needed", packed_bytes,
                    packed_bytes_of(layout, N, K));
    return hip_status(bitnet::launch_pack_elut(elut_format(layout), Wq, (int)N, (int)K, packed, (hipStream_t)stream),
                      "bitnet_pack_int_weights launch");
}

bitnet_status bitnet_quantize_act(const float* x, int64_t M, int64_t K, int8_t* xq, float* x_scale,
                                  int32_t* x_rowsum, void* stream) {
    if (!x || !xq || !x_scale) return fail(BITNET_E_INVALID, "null pointer argument");
    if (M < 1 || M > ((int64_t)1 << 31) - 1 || K < 1 || K > ((int64_t)1 << 20))
        return fail(BITNET_E_SHAPE, "need M >= 1 and 1 <= K <= 1048576; got M=%lld K=%lld", (long long)M,
                    (long long)K);
    if (!aligned(x, 16) || !aligned(xq, 16) || !aligned(x_scale, 4) || !aligned(x_rowsum, 4))
        return fail(BITNET_E_ALIGN, "x and xq need 16-byte alignment, x_scale and x_rowsum 4-byte");
    return hip_status(bitnet::launch_quantize_act(x, M, K, xq, x_scale, x_rowsum, (hipStream_t)stream),
                      "bitnet_quantize_act launch");
}

size_t bitnet_mpgemm_workspace_bytes(int layout, int64_t M, int64_t N, int64_t K) {
    if (!layout_ok(layout) || !layout_shape_ok(layout, N, K) || M < 1) return 0;
    if (layout == BITNET_LAYOUT_I2S && M > kDecodeMaxTokens)
        return bitnet::prefill_workspace_bytes(one_linear(nullptr, nullptr, N, nullptr, nullptr), M, K);
    if ((layout == BITNET_LAYOUT_TL2 || layout == BITNET_LAYOUT_TL1) && tl2_via_i2s(M, N, K))
        return align256((size_t)N * (size_t)K / 4) +
               bitnet::prefill_workspace_bytes(one_linear(nullptr, nullptr, N, nullptr, nullptr), M, K);
    return 0;
}

size_t bitnet_mpgemm_fused_workspace_bytes(int layout, int n_linears, const int64_t* N, int64_t K, int64_t M) {
    if (!layout_ok(layout) || !N || n_linears < 1 || n_linears > bitnet::kMaxFused || M < 1) return 0;
    for (int i = 0; i < n_linears; ++i)
        if (!layout_shape_ok(layout, N[i], K)) return 0;
    size_t need = 0;
    for (int i = 0; i < n_linears; ++i) {
        const size_t w = bitnet_mpgemm_workspace_bytes(layout, M, N[i], K);
        need = w > need ? w : need;
    }
    const bool tl2_gemm = (layout == BITNET_LAYOUT_TL2 || layout == BITNET_LAYOUT_TL1) && M > kDecodeMaxTokens;
    bool via = tl2_gemm;
    for (int i = 0; i < n_linears; ++i) via = via && tl2_via_i2s(M, N[i], K);
    if ((layout == BITNET_LAYOUT_I2S && M > kDecodeMaxTokens) || via) {
        bitnet::FusedLinears L{};
        L.count = n_linears;
        size_t words = 0;
        for (int i = 0; i < n_linears; ++i) {
            L.N[i] = (int)N[i];
            if (via) words += align256((size_t)N[i] * (size_t)K / 4);
        }
        bitnet::seal_fused(L);
        const size_t split = words + bitnet::prefill_workspace_bytes(L, M, K);
        need = split > need ? split : need;
    }
    return need;
}

}  // extern "C"

namespace {

// Checks of bitnet_mpgemm's arguments other than the workspace; sets *need to its workspace bytes.
bitnet_status mpgemm_check(int layout, const void* packed, size_t packed_bytes, const float* w_scale, int64_t N,
                           int64_t K, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum, int64_t M,
                           float* y, int32_t* acc, size_t* need) {
    if (!layout_ok(layout)) return fail(BITNET_E_LAYOUT, "unknown layout %d", layout);
    if (!packed || !w_scale || !xq || !x_scale || !y) return fail(BITNET_E_INVALID, "null pointer argument");
    if (!layout_shape_ok(layout, N, K))
        return fail(BITNET_E_SHAPE, "need N %% 16 == 0, K %% %d == 0, 0 < K <= %lld; got N=%lld K=%lld",
                    layout == BITNET_LAYOUT_C3G5 ? 320 : 64, (long long)kMaxK, (long long)N, (long long)K);
    if (M < 1 || M > ((int64_t)1 << 24)) return fail(BITNET_E_SHAPE, "need 1 <= M <= 2^24; got M=%lld", (long long)M);
    if (elut_layout(layout) && (uint64_t)N * (uint64_t)K >= ((uint64_t)1 << 32))
        return fail(BITNET_E_SHAPE, "integer-weight layouts need N*K below 2^32");
    if (!aligned(packed, 16) || !aligned(xq, 16) || !aligned(y, 16) || (acc && !aligned(acc, 16)) ||
        !aligned(w_scale, 4) || !aligned(x_scale, 4) || !aligned(x_rowsum, 4))
        return fail(BITNET_E_ALIGN, "packed, xq, y, acc and ws need 16-byte alignment, scales and x_rowsum 4-byte");
    if (packed_bytes < packed_bytes_of(layout, N, K))
        return fail(BITNET_E_INVALID, "packed buffer holds %zu bytes, %zu needed", packed_bytes,
                    packed_bytes_of(layout, N, K));
    if (i2s_tiled(layout) && ((uint64_t)N * (uint64_t)K >= ((uint64_t)1 << 32) ||
                              (uint64_t)M * (uint64_t)K >= ((uint64_t)1 << 32)))
        return fail(BITNET_E_SHAPE, "I2_S and TL1 need N*K and M*K below 2^32; got M=%lld N=%lld K=%lld",
                    (long long)M, (long long)N, (long long)K);
    *need = bitnet_mpgemm_workspace_bytes(layout, M, N, K);
    return BITNET_OK;
}

// The launches of bitnet_mpgemm once its arguments are checked (ws holds at least the workspace it needs).
bitnet_status mpgemm_run(int layout, const void* packed, size_t packed_bytes, const float* w_scale, int64_t N,
                         int64_t K, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum, int64_t M,
                         float* y, int32_t* acc, void* ws, size_t ws_bytes, hipStream_t s) {
    (void)packed_bytes;
    if (lossy_layout(layout)) {
        // TL2_0 / TL1_0: table lookups on int8-quantised tables; one token on the persistent table kernels (every
        // work group builds the row's tables once), else slices of 8 tokens
        if (layout == BITNET_LAYOUT_TL2_0 && M == 1 && bitnet::tl2_stream_fits((int)K))
            return hip_status(bitnet::launch_tl2_stream(one_linear(packed, w_scale, N, y, acc), nullptr, (int)K,
                                                        const_cast<int8_t*>(xq), const_cast<float*>(x_scale), nullptr,
                                                        s, true),
                              "bitnet_mpgemm launch");
        if (layout == BITNET_LAYOUT_TL1_0 && M == 1 && bitnet::tl1_stream_fits((int)K))
            return hip_status(bitnet::launch_tl1_lossy_stream(one_linear(packed, w_scale, N, y, acc), nullptr, (int)K,
                                                              const_cast<int8_t*>(xq), const_cast<float*>(x_scale),
                                                              nullptr, s),
                              "bitnet_mpgemm launch");
        return hip_status(lookup_sliced(layout == BITNET_LAYOUT_TL1_0, true, one_linear(packed, w_scale, N, y, acc),
                                        xq, x_scale, M, K, s),
                          "bitnet_mpgemm launch");
    }
    if (elut_layout(layout))   // table lookups of the integer-weight formats, any M (slices of 2 or 4 tokens)
        return hip_status(bitnet::launch_elut_generic(elut_format(layout), one_linear(packed, w_scale, N, y, acc), nullptr,
                                                      xq, x_scale, (int)M, (int)K, nullptr, nullptr, nullptr, s),
                          "bitnet_mpgemm launch");
    if (i2s_tiled(layout) && (M <= kDecodeMaxTokens || bitnet::i2s_sliced_ok(M, K, x_rowsum != nullptr)))
        return hip_status(bitnet::launch_i2s_decode(one_linear(packed, w_scale, N, y, acc), xq, x_scale, x_rowsum,
                                                    (int)M, (int)K, s, word_format(layout)),
                          "bitnet_mpgemm launch");
    if (layout == BITNET_LAYOUT_TL1) {
        // the TL1 words rewritten as I2_S words at the start of the workspace, the GEMM's split-K slices after them
        const size_t wbytes = align256((size_t)N * (size_t)K / 4);
        const int n1 = (int)N;
        void* dst = ws;
        hipError_t e = bitnet::launch_tl1_to_i2s(&packed, &n1, &dst, 1, (int)K, s);
        if (e == hipSuccess)
            e = bitnet::launch_i2s_prefill(one_linear(ws, w_scale, N, y, acc), xq, x_scale, x_rowsum, (int)M, (int)K,
                                           static_cast<uint8_t*>(ws) + wbytes, ws_bytes - wbytes, s);
        return hip_status(e, "bitnet_mpgemm launch");
    }
    if (layout == BITNET_LAYOUT_I2S)
        return hip_status(bitnet::launch_i2s_prefill(one_linear(packed, w_scale, N, y, acc), xq, x_scale, x_rowsum,
                                                     (int)M, (int)K, ws, ws_bytes, s),
                          "bitnet_mpgemm launch");
    if (M == 1 && bitnet::tl2_stream_fits((int)K))
        return hip_status(bitnet::launch_tl2_stream(one_linear(packed, w_scale, N, y, acc), nullptr, (int)K,
                                                    const_cast<int8_t*>(xq), const_cast<float*>(x_scale), nullptr, s),
                          "bitnet_mpgemm launch");
    if (tl2_via_i2s(M, N, K)) {
        // the weights in the I2_S layout at the start of the workspace, the GEMM's split-K slices after them
        const size_t wbytes = align256((size_t)N * (size_t)K / 4);
        const int n1 = (int)N;
        void* dst = ws;
        hipError_t e = bitnet::launch_tl2_to_i2s(&packed, &n1, &dst, 1, (int)K, s);
        if (e == hipSuccess)
            e = bitnet::launch_i2s_prefill(one_linear(ws, w_scale, N, y, acc), xq, x_scale, x_rowsum, (int)M, (int)K,
                                           static_cast<uint8_t*>(ws) + wbytes, ws_bytes - wbytes, s);
        return hip_status(e, "bitnet_mpgemm launch");
    }
    if (bitnet::tl2_mfma_max_tokens((int)K) > 0)
        return hip_status(bitnet::launch_tl2_mfma_decode(one_linear(packed, w_scale, N, y, acc), xq, x_scale, (int)M,
                                                         (int)K, s),
                          "bitnet_mpgemm launch");
    return hip_status(lookup_sliced(false, false, one_linear(packed, w_scale, N, y, acc), xq, x_scale, M, K, s),
                      "bitnet_mpgemm launch");
}

// Scratch of bitnet_mpgemm_noalloc: one copy of this array on every GPU the library runs on, held until the
// process ends.  In host code its name is only a handle; the device address of each GPU's copy comes from
// hipGetSymbolAddress (once per device, with that device current) and is the only form passed to kernels.
constexpr size_t kNoallocScratchBytes = BITNET_NOALLOC_SCRATCH_BYTES;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

}  // namespace

static __device__ __align__(256) uint8_t scratch[kNoallocScratchBytes];

namespace {

// The current device's copy of `scratch`.
bitnet_status scratch_on_current_device(void** out) {
    int dev = -1;
    const hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_status(e, "hipGetDevice");
    if (dev < 0 || dev >= kMaxDevices) return fail(BITNET_E_HIP, "device %d outside the supported range", dev);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_ptr[dev]) {
        void* p = nullptr;
        const hipError_t g = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (g != hipSuccess || !p) return hip_status(g != hipSuccess ? g : hipErrorInvalidSymbol,
                                                     "hipGetSymbolAddress of the no-allocation scratch");
        g_scratch_ptr[dev] = p;
    }
    *out = g_scratch_ptr[dev];
    return BITNET_OK;
}

}  // namespace

extern "C" {

bitnet_status bitnet_mpgemm(int layout, const void* packed, size_t packed_bytes, const float* w_scale, int64_t N,
                            int64_t K, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum, int64_t M,
                            float* y, int32_t* acc, void* ws, size_t ws_bytes, void* stream) {
    size_t need = 0;
    const bitnet_status st = mpgemm_check(layout, packed, packed_bytes, w_scale, N, K, xq, x_scale, x_rowsum, M, y,
                                          acc, &need);
    if (st != BITNET_OK) return st;
    if (!aligned(ws, 16)) return fail(BITNET_E_ALIGN, "ws needs 16-byte alignment");
    // the workspace holds split-K slices of the prefill GEMM (used when x_rowsum is given) and TL2 weights
    // rewritten for it
    if (need && (!ws || ws_bytes < need)) return fail(BITNET_E_WORKSPACE, "mpgemm workspace needs %zu bytes", need);
    return mpgemm_run(layout, packed, packed_bytes, w_scale, N, K, xq, x_scale, x_rowsum, M, y, acc, ws, ws_bytes,
                      (hipStream_t)stream);
}

bitnet_status bitnet_mpgemm_noalloc(int layout, const void* packed, size_t packed_bytes, const float* w_scale,
                                    int64_t N, int64_t K, const int8_t* xq, const float* x_scale,
                                    const int32_t* x_rowsum, int64_t M, float* y, int32_t* acc, void* stream) {
    size_t need = 0;
    bitnet_status st = mpgemm_check(layout, packed, packed_bytes, w_scale, N, K, xq, x_scale, x_rowsum, M, y, acc,
                                    &need);
    if (st != BITNET_OK) return st;
    if (need > kNoallocScratchBytes)
        return fail(BITNET_E_WORKSPACE, "this shape needs %zu bytes of workspace; the no-allocation scratch holds %zu",
                    need, kNoallocScratchBytes);
    void* ws = nullptr;
    if (need) {
        st = scratch_on_current_device(&ws);
        if (st != BITNET_OK) return st;
    }
    return mpgemm_run(layout, packed, packed_bytes, w_scale, N, K, xq, x_scale, x_rowsum, M, y, acc, ws,
                      need ? kNoallocScratchBytes : 0, (hipStream_t)stream);
}

bitnet_status bitnet_mpgemm_fused(int layout, int n_linears, const void* const* packed, const size_t* packed_bytes,
                                  const float* const* w_scale, const int64_t* N, int64_t K, const float* x, int64_t M,
                                  int8_t* xq, float* x_scale, int32_t* x_rowsum, float* const* y, void* ws,
                                  size_t ws_bytes, void* stream) {
    if (!layout_ok(layout)) return fail(BITNET_E_LAYOUT, "unknown layout %d", layout);
    if (n_linears < 1 || n_linears > bitnet::kMaxFused)
        return fail(BITNET_E_INVALID, "n_linears must be 1..%d; got %d", bitnet::kMaxFused, n_linears);
    if (!packed || !packed_bytes || !w_scale || !N || !y || !xq || !x_scale || !x_rowsum)
        return fail(BITNET_E_INVALID, "null pointer argument");
    const bool quantise = x != nullptr;       // NULL x: xq, x_scale and x_rowsum already hold the activation
    if (M < 1 || M > ((int64_t)1 << 24)) return fail(BITNET_E_SHAPE, "need 1 <= M <= 2^24; got M=%lld", (long long)M);
    if (!aligned(x, 16) || !aligned(xq, 16) || !aligned(x_scale, 4) || !aligned(x_rowsum, 4))
        return fail(BITNET_E_ALIGN, "x and xq need 16-byte alignment, x_scale and x_rowsum 4-byte");
    size_t need = 0;
    for (int i = 0; i < n_linears; ++i) {
        if (!packed[i] || !w_scale[i] || !y[i]) return fail(BITNET_E_INVALID, "null pointer for weight %d", i);
        if (!layout_shape_ok(layout, N[i], K))
            return fail(BITNET_E_SHAPE, "weight %d: need N %% 16 == 0, K %% %d == 0, 0 < K <= %lld; got N=%lld K=%lld", i,
                        layout == BITNET_LAYOUT_C3G5 ? 320 : 64, (long long)kMaxK, (long long)N[i], (long long)K);
        if (!aligned(packed[i], 16) || !aligned(y[i], 16) || !aligned(w_scale[i], 4))
            return fail(BITNET_E_ALIGN, "weight %d: packed and y need 16-byte alignment, w_scale 4-byte", i);
        if (packed_bytes[i] < packed_bytes_of(layout, N[i], K))
            return fail(BITNET_E_INVALID, "weight %d: packed buffer holds %zu bytes, %zu needed", i, packed_bytes[i],
                        packed_bytes_of(layout, N[i], K));
        if (i2s_tiled(layout) && ((uint64_t)N[i] * (uint64_t)K >= ((uint64_t)1 << 32) ||
                                  (uint64_t)M * (uint64_t)K >= ((uint64_t)1 << 32)))
            return fail(BITNET_E_SHAPE, "weight %d: I2_S and TL1 need N*K and M*K below 2^32", i);
        const size_t w = bitnet_mpgemm_workspace_bytes(layout, M, N[i], K);
        need = w > need ? w : need;
    }
    // a fused prefill launch splits K only where ws holds the slices of all its weights; the largest single
    // workspace is always enough for the call to run
    if (need && (!ws || ws_bytes < need)) return fail(BITNET_E_WORKSPACE, "workspace needs %zu bytes", need);
    if (!aligned(ws, 16)) return fail(BITNET_E_ALIGN, "ws needs 16-byte alignment");

    hipStream_t s = (hipStream_t)stream;
    if (elut_layout(layout) || lossy_layout(layout)) {
        // every weight of the group in one table-lookup launch; one token quantised inside it, else the quantiser
        // first (TL2_0 and TL1_0: launches of up to 8 tokens)
        bitnet::FusedLinears L{};
        L.count = n_linears;
        int64_t rgs = 0;
        for (int i = 0; i < n_linears; ++i) {
            L.packed[i] = static_cast<const uint8_t*>(packed[i]);
            L.w_scale[i] = w_scale[i];
            L.y[i] = y[i];
            L.acc[i] = nullptr;
            L.N[i] = (int)N[i];
            rgs += N[i] / bitnet::kRowsPerGroup;
        }
        if (rgs > ((int64_t)1 << 26)) return fail(BITNET_E_SHAPE, "too many output rows in one launch");
        bitnet::seal_fused(L);
        const bool tl1 = layout == BITNET_LAYOUT_TL1_0;
        if (layout == BITNET_LAYOUT_TL2_0 && M == 1 && bitnet::tl2_stream_fits((int)K))
            // one token: the persistent table kernel (the row quantised inside when x is given)
            return hip_status(bitnet::launch_tl2_stream(L, quantise ? x : nullptr, (int)K, xq, x_scale, x_rowsum, s,
                                                        true),
                              "bitnet_mpgemm_fused launch");
        if (layout == BITNET_LAYOUT_TL1_0 && M == 1 && bitnet::tl1_stream_fits((int)K))
            return hip_status(bitnet::launch_tl1_lossy_stream(L, quantise ? x : nullptr, (int)K, xq, x_scale, x_rowsum,
                                                              s),
                              "bitnet_mpgemm_fused launch");
        if (quantise && M == 1) {
            const hipError_t e =
                lossy_layout(layout)
                    ? (tl1 ? bitnet::launch_tl1_elut_decode(L, x, nullptr, nullptr, 1, (int)K, xq, x_scale, x_rowsum, s,
                                                            true)
                           : bitnet::launch_tl2_elut_decode(L, x, nullptr, nullptr, 1, (int)K, xq, x_scale, x_rowsum, s,
                                                            true))
                    : bitnet::launch_elut_generic(elut_format(layout), L, x, nullptr, nullptr, 1, (int)K, xq, x_scale,
                                                  x_rowsum, s);
            return hip_status(e, "bitnet_mpgemm_fused launch");
        }
        hipError_t e = quantise ? bitnet::launch_quantize_act(x, M, K, xq, x_scale, x_rowsum, s) : hipSuccess;
        if (e == hipSuccess)
            e = lossy_layout(layout) ? lookup_sliced(tl1, true, L, xq, x_scale, M, K, s)
                                     : bitnet::launch_elut_generic(elut_format(layout), L, nullptr, xq, x_scale, (int)M,
                                                                   (int)K, nullptr, nullptr, nullptr, s);
        return hip_status(e, "bitnet_mpgemm_fused launch");
    }
    // the small-batch regime (17..128 tokens, K <= 16384): the decode GEMV in token slices, for I2_S and TL1
    const bool sliced = i2s_tiled(layout) && bitnet::i2s_sliced_ok(M, K, true);
    if (layout == BITNET_LAYOUT_I2S || (layout == BITNET_LAYOUT_TL1 && (M <= kDecodeMaxTokens || sliced))) {
        const int fmt = word_format(layout);
        bitnet::FusedLinears L{};
        L.count = n_linears;
        int64_t rgs = 0;
        for (int i = 0; i < n_linears; ++i) {
            L.packed[i] = static_cast<const uint8_t*>(packed[i]);
            L.w_scale[i] = w_scale[i];
            L.y[i] = y[i];
            L.acc[i] = nullptr;
            L.N[i] = (int)N[i];
            rgs += N[i] / bitnet::kRowsPerGroup;
        }
        if (rgs > ((int64_t)1 << 30)) return fail(BITNET_E_SHAPE, "too many output rows in one launch");
        bitnet::seal_fused(L);
        if (quantise && M == 1 && K <= bitnet::kFusedMaxK)   // one launch: quantise inside every work group
            return hip_status(bitnet::launch_i2s_gemv1_stream(L, x, (int)K, xq, x_scale, x_rowsum, s, fmt),
                              "bitnet_mpgemm_fused launch");
        hipError_t e = quantise ? bitnet::launch_quantize_act(x, M, K, xq, x_scale, x_rowsum, s) : hipSuccess;
        if (e == hipSuccess)
            e = (M <= kDecodeMaxTokens || sliced)
                    ? bitnet::launch_i2s_decode(L, xq, x_scale, x_rowsum, (int)M, (int)K, s, fmt)
                    : bitnet::launch_i2s_prefill(L, xq, x_scale, x_rowsum, (int)M, (int)K, ws, ws_bytes, s);
        return hip_status(e, "bitnet_mpgemm_fused launch");
    }
    // TL2: one token: one launch for every weight that quantises inside (the MFMA expansion, or the table lookups
    // where the whole row's tables fit in LDS).  Otherwise the quantiser once, then one MFMA launch for every weight
    // (token slices that fit in LDS) or, where that path does not cover K, one table-lookup launch per weight.
    // TL2 and TL1 past 16 tokens: the quantiser, every weight rewritten in the I2_S layout, one prefill launch.
    bitnet::FusedLinears L{};
    L.count = n_linears;
    int64_t rgs = 0;
    for (int i = 0; i < n_linears; ++i) {
        L.packed[i] = static_cast<const uint8_t*>(packed[i]);
        L.w_scale[i] = w_scale[i];
        L.y[i] = y[i];
        L.acc[i] = nullptr;
        L.N[i] = (int)N[i];
        rgs += N[i] / bitnet::kRowsPerGroup;
    }
    if (rgs > ((int64_t)1 << 30)) return fail(BITNET_E_SHAPE, "too many output rows in one launch");
    bitnet::seal_fused(L);
    const bool tl2 = layout == BITNET_LAYOUT_TL2;
    if (tl2 && M == 1 && quantise && bitnet::tl2_mfma_quant_fits((int)K))
        return hip_status(bitnet::launch_tl2_mfma_quant(L, x, (int)K, xq, x_scale, x_rowsum, s),
                          "bitnet_mpgemm_fused launch");
    if (tl2 && M == 1 && bitnet::tl2_stream_fits((int)K)) {
        if (!quantise) return hip_status(bitnet::launch_tl2_stream(L, nullptr, (int)K, xq, x_scale, x_rowsum, s),
                                         "bitnet_mpgemm_fused launch");
        return hip_status(bitnet::launch_tl2_stream(L, x, (int)K, xq, x_scale, x_rowsum, s),
                          "bitnet_mpgemm_fused launch");
    }
    hipError_t e = quantise ? bitnet::launch_quantize_act(x, M, K, xq, x_scale, x_rowsum, s) : hipSuccess;
    if (e != hipSuccess) return hip_status(e, "bitnet_mpgemm_fused launch");
    // more than 16 tokens: every weight rewritten in the I2_S layout, then one prefill launch for all of them, where
    // the workspace holds all the rewritten weights (else one bitnet_mpgemm per weight, below)
    bool via = M > kDecodeMaxTokens;
    size_t words = 0;
    for (int i = 0; i < n_linears; ++i) {
        via = via && tl2_via_i2s(M, N[i], K);
        words += align256((size_t)N[i] * (size_t)K / 4);
    }
    if (via && ws_bytes >= words) {
        bitnet::FusedLinears T = L;
        size_t off = 0;
        void* dst[bitnet::kMaxFused];
        int n32[bitnet::kMaxFused];
        for (int i = 0; i < n_linears; ++i) {
            dst[i] = static_cast<uint8_t*>(ws) + off;
            n32[i] = (int)N[i];
            T.packed[i] = static_cast<const uint8_t*>(dst[i]);
            off += align256((size_t)N[i] * (size_t)K / 4);
        }
        e = tl2 ? bitnet::launch_tl2_to_i2s(packed, n32, dst, n_linears, (int)K, s)
                : bitnet::launch_tl1_to_i2s(packed, n32, dst, n_linears, (int)K, s);
        if (e == hipSuccess)
            e = bitnet::launch_i2s_prefill(T, xq, x_scale, x_rowsum, (int)M, (int)K, static_cast<uint8_t*>(ws) + words,
                                           ws_bytes - words, s);
        return hip_status(e, "bitnet_mpgemm_fused launch");
    }
    if (tl2 && M <= kDecodeMaxTokens && bitnet::tl2_mfma_max_tokens((int)K) > 0)
        return hip_status(bitnet::launch_tl2_mfma_decode(L, xq, x_scale, (int)M, (int)K, s),
                          "bitnet_mpgemm_fused launch");
    for (int i = 0; i < n_linears; ++i) {
        const bitnet_status st = bitnet_mpgemm(layout, packed[i], packed_bytes[i], w_scale[i], N[i], K, xq, x_scale,
                                               x_rowsum, M, y[i], nullptr, ws, ws_bytes, stream);
        if (st != BITNET_OK) return st;
    }
    return ok();
}

bitnet_status bitnet_elut_tables(const int8_t* xq, int64_t M, int64_t K, int16_t* lut, int16_t* lut1, void* stream) {
    if (!xq || !lut) return fail(BITNET_E_INVALID, "null pointer argument");
    if (M < 1 || M > ((int64_t)1 << 24) || K <= 0 || K % bitnet::kSubK != 0 || K > kMaxK)
        return fail(BITNET_E_SHAPE, "need M >= 1 and K %% 64 == 0, 0 < K <= %lld; got M=%lld K=%lld", (long long)kMaxK,
                    (long long)M, (long long)K);
    const int64_t three = (K / bitnet::kTl2BlockK) * bitnet::kTl2BlockK;
    if (three == 0) return fail(BITNET_E_SHAPE, "K = %lld has no 384-weight TL2 block", (long long)K);
    if (K != three && !lut1) return fail(BITNET_E_INVALID, "lut1 is required when K %% 384 != 0");
    if (!aligned(xq, 16) || !aligned(lut, 16) || (lut1 && !aligned(lut1, 16)))
        return fail(BITNET_E_ALIGN, "xq, lut and lut1 need 16-byte alignment");
    return hip_status(bitnet::launch_elut_tables(xq, (int)M, (int)K, lut, lut1, (hipStream_t)stream),
                      "bitnet_elut_tables launch");
}

const char* bitnet_status_string(int status) {
    switch (status) {
        case BITNET_OK: return "ok";
        case BITNET_E_INVALID: return "invalid argument";
        case BITNET_E_SHAPE: return "unsupported shape";
        case BITNET_E_ALIGN: return "misaligned pointer";
        case BITNET_E_LAYOUT: return "unknown or unavailable layout";
        case BITNET_E_WORKSPACE: return "workspace missing or too small";
        case BITNET_E_HIP: return "HIP runtime error";
        default: return "unknown status";
    }
}

const char* bitnet_last_error(void) { return g_last_error; }

}  // extern "C"
