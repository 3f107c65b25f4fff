// Internal declarations shared by the library's translation units (host launchers + device helpers).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace bitnet {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

constexpr int kRowsPerGroup = 16;     // weight rows per MFMA tile (both layouts)
constexpr int kSubK = 64;             // k per 16x16x64 int8 MFMA
constexpr int kI2sBlockK = 256;       // I2_S block: up to four 64-k sub-tiles, 1 KiB per row group
constexpr int kTl2BlockK = 384;       // TL2 block BK3: 128 triples per row
constexpr int kNumXcd = 8;            // MI355X: 8 accelerator dies, work groups dealt round-robin

// ------------------------------------------------------------------------------------------------
// Device helpers
// ------------------------------------------------------------------------------------------------

// Work groups are dealt to the XCDs round-robin by id.  Renumber them so that each XCD owns one
// contiguous range of logical ids; neighbouring tiles (split-K siblings) then share an L2.
__device__ __forceinline__ int xcd_logical_id(int bid, int nblocks) {
    const int per = nblocks / kNumXcd, extra = nblocks % kNumXcd;
    const int xcd = bid % kNumXcd, idx = bid / kNumXcd;
    return xcd * per + (xcd < extra ? xcd : extra) + idx;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
    return v;
}

// Reductions over the 64 lanes of a wave, the result in every lane: DPP steps inside each row of 16 lanes
// (swap neighbours, swap pairs, rotate the row by 4 and by 8), then the four row results read as scalars.
__device__ __forceinline__ int dpp_row_step(int v, int ctrl_sel) {
    switch (ctrl_sel) {
        case 0: return __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xF, 0xF, false);   // quad_perm [1, 0, 3, 2]
        case 1: return __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xF, 0xF, false);   // quad_perm [2, 3, 0, 1]
        case 2: return __builtin_amdgcn_update_dpp(0, v, 0x124, 0xF, 0xF, false);  // row_ror:4
        default: return __builtin_amdgcn_update_dpp(0, v, 0x128, 0xF, 0xF, false); // row_ror:8
    }
}

__device__ __forceinline__ float wave_max_all(float v) {
#pragma unroll
    for (int i = 0; i < 4; ++i) v = fmaxf(v, __int_as_float(dpp_row_step(__float_as_int(v), i)));
    const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 0));
    const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 16));
    const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 32));
    const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), 48));
    return fmaxf(fmaxf(r0, r1), fmaxf(r2, r3));
}

__device__ __forceinline__ int wave_sum_all(int v) {
#pragma unroll
    for (int i = 0; i < 4; ++i) v += dpp_row_step(v, i);
    return __builtin_amdgcn_readlane(v, 0) + __builtin_amdgcn_readlane(v, 16) + __builtin_amdgcn_readlane(v, 32) +
           __builtin_amdgcn_readlane(v, 48);
}

// Lanes of one wave hand data to other lanes of the same wave through LDS: the writes are ordered before the
// reads by a release/acquire pair at work-group scope restricted to LDS (it waits for the wave's LDS operations
// only, never for its global loads in flight) around a wave barrier, which also keeps the compiler from moving
// the reads above the writes.  No other wave reads the data, so no work-group barrier is needed.
__device__ __forceinline__ void wave_lds_handoff() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// int8 codes of four activations, packed little-endian: clamp(rint(fp32(x * s)), -128, 127) (Sec. 2.1).
// rint gives an integer-valued float; + 128 is exact; v_cvt_pk_u8_f32 then converts it exactly (saturating
// to [0, 255], which is the clamp) into its byte, and XOR 0x80 turns the offset byte into two's complement.
__device__ __forceinline__ uint32_t quant4(float4 v, float s) {
    uint32_t p = __builtin_amdgcn_cvt_pk_u8_f32(rintf(v.x * s) + 128.0f, 0, 0u);
    p = __builtin_amdgcn_cvt_pk_u8_f32(rintf(v.y * s) + 128.0f, 1, p);
    p = __builtin_amdgcn_cvt_pk_u8_f32(rintf(v.z * s) + 128.0f, 2, p);
    p = __builtin_amdgcn_cvt_pk_u8_f32(rintf(v.w * s) + 128.0f, 3, p);
    return p ^ 0x80808080u;
}

// sum of the four signed bytes of a word, added to acc
__device__ __forceinline__ int byte_sum4(uint32_t w, int acc) {
    return __builtin_amdgcn_sdot4((int)w, 0x01010101, acc, false);
}

// The four int8 codes of k = 4f .. 4f+3 sit in field f (bits 2f, 2f+1) of the four bytes of an I2_S word.
__device__ __forceinline__ v4i unpack_codes(uint32_t w) {
    v4i b;
    b.x = (int)(w & 0x03030303u);
    b.y = (int)((w >> 2) & 0x03030303u);
    b.z = (int)((w >> 4) & 0x03030303u);
    b.w = (int)((w >> 6) & 0x03030303u);
    return b;
}

// Weight formats that share the I2_S tiling (one 32-bit word = 16 weights of one row, k = 16 q + e, e = 0..15):
// I2_S words hold 2-bit codes t + 1; TL1 words hold the Table 5 codes c = 3 (t0 + 1) + (t1 + 1) of 8 pairs, pair i
// (weights e = 2i, 2i + 1) in byte i % 4, low nibble for i < 4 and high nibble for i >= 4.
constexpr int kFmtI2s = 0;
constexpr int kFmtTl1 = 1;

// A TL1 word as the offset codes t + 1 of its 16 weights, in four int8 words:
// [t0 + 1 of pairs 0..3, t1 + 1 of pairs 0..3, t0 + 1 of pairs 4..7, t1 + 1 of pairs 4..7], which are the weights
// e = 0,2,4,6 | 1,3,5,7 | 8,10,12,14 | 9,11,13,15.  floor(c / 3) = (11 c) >> 5 for c <= 8, and every byte of the
// word products stays below 256, so the word arithmetic never carries from one byte into the next.
__device__ __forceinline__ v4i tl1_codes(uint32_t w) {
    const uint32_t lo = w & 0x0F0F0F0Fu, hi = (w >> 4) & 0x0F0F0F0Fu;
    const uint32_t qlo = ((lo * 11u) >> 5) & 0x07070707u, qhi = ((hi * 11u) >> 5) & 0x07070707u;
    v4i b;
    b.x = (int)qlo;
    b.y = (int)(lo - 3u * qlo);
    b.z = (int)qhi;
    b.w = (int)(hi - 3u * qhi);
    return b;
}

// The 16 activation codes of k = 16 q .. 16 q + 15 (natural order in) in the order tl1_codes gives the weights.
// v_perm_b32 picks byte s of {hi, lo} (s < 4: lo) for every selector byte s.
__device__ __forceinline__ v4i tl1_perm16(v4i a) {
    v4i o;
    o.x = (int)__builtin_amdgcn_perm((uint32_t)a.y, (uint32_t)a.x, 0x06040200u);
    o.y = (int)__builtin_amdgcn_perm((uint32_t)a.y, (uint32_t)a.x, 0x07050301u);
    o.z = (int)__builtin_amdgcn_perm((uint32_t)a.w, (uint32_t)a.z, 0x06040200u);
    o.w = (int)__builtin_amdgcn_perm((uint32_t)a.w, (uint32_t)a.z, 0x07050301u);
    return o;
}

// The MFMA B operand (offset codes) of one packed word, and the A operand order that matches it.
template <int FMT>
__device__ __forceinline__ v4i decode_b(uint32_t w) {
    if constexpr (FMT == kFmtTl1) return tl1_codes(w);
    else return unpack_codes(w);
}
template <int FMT>
__device__ __forceinline__ v4i order_a(v4i a) {
    if constexpr (FMT == kFmtTl1) return tl1_perm16(a);
    else return a;
}

__device__ __forceinline__ uint32_t word_of(const v4u& v, int j) {
    return j == 0 ? v.x : j == 1 ? v.y : j == 2 ? v.z : v.w;
}

__device__ __forceinline__ v4u load_stream16(const uint8_t* p) {
    return __builtin_nontemporal_load(reinterpret_cast<const v4u*>(p));
}

__device__ __forceinline__ v4i mfma16x16x64(v4i a, v4i b, v4i c) {
    return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// ------------------------------------------------------------------------------------------------
// Host launchers (each returns the launch status; shapes were validated by the caller)
// ------------------------------------------------------------------------------------------------
hipError_t launch_quantize_act(const float* x, int64_t M, int64_t K, int8_t* xq, float* x_scale,
                               int32_t* x_rowsum, hipStream_t stream);

size_t pack_workspace_bytes();
hipError_t launch_pack(int layout, const float* W, int64_t N, int64_t K, void* packed, float* w_scale,
                       void* ws, hipStream_t stream);

constexpr int kMaxSplits = 16;
int device_cus();

// Up to kMaxFused weights that read the same activation, served by one decode launch.
constexpr int kMaxFused = 8;
struct FusedLinears {
    const uint8_t* packed[kMaxFused];
    const float* w_scale[kMaxFused];
    float* y[kMaxFused];
    int32_t* acc[kMaxFused];       // optional exact accumulators (NULL entries allowed)
    int N[kMaxFused];
    int rg_start[kMaxFused + 1];   // first 16-row group of each weight in the launch; INT_MAX past the last
    int count;
    int total;                     // row groups in the launch
};

// Which weight the launch's row group g belongs to, and its row group within that weight.  The bounds are
// increasing (INT_MAX past the last weight), so a compare-and-select chain over the fixed maximum finds it; for a
// uniform g it is all scalar.
__device__ __forceinline__ void locate(const FusedLinears& L, int g, int& li, int& rg) {
    int l = 0, start = 0;
#pragma unroll
    for (int i = 1; i < kMaxFused; ++i) {
        const int st = L.rg_start[i];
        l = g >= st ? i : l;
        start = g >= st ? st : start;
    }
    li = l;
    rg = g - start;
}

template <typename T>
__device__ __forceinline__ T pick(const T (&a)[kMaxFused], int li) {
    T v = a[0];
#pragma unroll
    for (int i = 1; i < kMaxFused; ++i) v = li == i ? a[i] : v;
    return v;
}

// Fill the launch totals once the first `count` entries are set.
inline void seal_fused(FusedLinears& L) {
    int64_t rgs = 0;
    for (int i = 0; i < L.count; ++i) {
        L.rg_start[i] = (int)rgs;
        rgs += L.N[i] / kRowsPerGroup;
    }
    L.total = (int)rgs;
    for (int i = L.count; i <= kMaxFused; ++i) L.rg_start[i] = i == L.count ? L.total : 0x7fffffff;
}
// Prefill (M > 16): one launch for up to kMaxFused weights that read the same activation; split-K over the
// workspace when it is given and large enough (and x_rowsum is given).
size_t prefill_workspace_bytes(const FusedLinears& L, int64_t M, int64_t K);
hipError_t launch_i2s_prefill(const FusedLinears& L, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum,
                              int M, int K, void* ws, size_t ws_bytes, hipStream_t stream);
constexpr int64_t kFusedMaxK = 61440;   // single-token fused quantise+GEMV keeps the K codes in LDS
// fmt: kFmtI2s or kFmtTl1 (the weights' word format; both formats share the I2_S tiling).  Up to 16 tokens; more
// (the small-batch regime) where i2s_sliced_ok holds: token slices of up to 16 in one launch.
constexpr int kSmallBatchMaxTokens = 112;   // from 128 tokens the prefill GEMM is as fast
inline bool i2s_sliced_ok(int64_t M, int64_t K, bool has_rowsum) {
    return M > 16 && M <= kSmallBatchMaxTokens && has_rowsum && K <= 16384;
}
hipError_t launch_i2s_decode(const FusedLinears& L, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum,
                             int M, int K, hipStream_t stream, int fmt = kFmtI2s);
hipError_t launch_i2s_gemv1_stream(const FusedLinears& L, const float* x, int K, int8_t* xq, float* x_scale,
                                   int32_t* x_rowsum, hipStream_t stream, int fmt = kFmtI2s);
// The TL1 weights of `count` (1..kMaxFused) N[i] x K tensors rewritten as I2_S words (same positions, N[i] K / 4
// bytes at i2s_out[i]), for the prefill GEMM; one launch.
hipError_t launch_tl1_to_i2s(const void* const* packed, const int* N, void* const* i2s_out, int count, int K,
                             hipStream_t stream);
constexpr int kElutMaxTokens = 8;     // tokens per ELUT launch
int tl2_elut_waves(int M);
size_t tl2_elut_lds_bytes(int M);
// The TL2 layout by table lookups, 1..8 tokens, every weight of L in one launch.  x NULL: xq and x_scale hold
// the M tokens' codes and scales.  x set (M == 1): the fp32 row is quantised inside the launch, which writes its
// codes, scale and code sum to xq_out, s_out and rs_out.  lossy: TL2_0 (Sec. 3.2.1), the tables quantised to int8
// per token and block before the lookups.
hipError_t launch_tl2_elut_decode(const FusedLinears& L, const float* x, const int8_t* xq, const float* x_scale,
                                  int M, int K, int8_t* xq_out, float* s_out, int32_t* rs_out, hipStream_t stream,
                                  bool lossy);
// The TL1 layout by table lookups (Algorithm TL1), arguments as above; lossy: TL1_0.
hipError_t launch_tl1_elut_decode(const FusedLinears& L, const float* x, const int8_t* xq, const float* x_scale,
                                  int M, int K, int8_t* xq_out, float* s_out, int32_t* rs_out, hipStream_t stream,
                                  bool lossy);
hipError_t launch_elut_tables(const int8_t* xq, int M, int K, int16_t* lut, int16_t* lut1, hipStream_t stream);
// One token, TL2, every weight of a group in one launch; x (fp32) is quantised inside, or, when x is NULL, xq is
// read.  Only where the whole row's tables fit in LDS (tl2_stream_fits); the caller falls back otherwise.
bool tl2_stream_fits(int K);
// Up to kTl2MfmaMaxTokens tokens per launch (already quantised), TL2 weights expanded to int8 for MFMA; every
// weight of a group in one launch.  tl2_mfma_max_tokens(K) is the slice one launch takes at this K (0: K has no
// 384-k block, or one token's codes do not fit in LDS); the launcher slices M itself.  Past 48 blocks a row group
// takes several batches.
constexpr int kTl2MfmaMaxTokens = 16;
int tl2_mfma_max_tokens(int K);
bool tl2_mfma_quant_fits(int K);      // launch_tl2_mfma_quant covers this K
hipError_t launch_tl2_mfma_decode(const FusedLinears& L, const int8_t* xq, const float* x_scale, int M, int K,
                                  hipStream_t stream);
hipError_t launch_tl2_mfma_quant(const FusedLinears& L, const float* x, int K, int8_t* xq, float* x_scale,
                                 int32_t* x_rowsum, hipStream_t stream);
// The TL2 weights of `count` (1..kMaxFused) N[i] x K tensors rewritten in the I2_S layout (N[i] K / 4 bytes at
// i2s_out[i]), for the prefill GEMM; one launch.
hipError_t launch_tl2_to_i2s(const void* const* packed, const int* N, void* const* i2s_out, int count, int K,
                             hipStream_t stream);
// One token, TL1_0, every weight of L in one launch: the whole row's int8 pair tables built once per work group
// (x set: the row quantised inside, as launch_tl2_stream).  Only where tl1_stream_fits(K).
bool tl1_stream_fits(int K);
hipError_t launch_tl1_lossy_stream(const FusedLinears& L, const float* x, int K, int8_t* xq, float* x_scale,
                                   int32_t* x_rowsum, hipStream_t stream);
// lossy: TL2_0 (Sec. 3.2.1), each block's tables quantised to int8 with its power-of-two scale.
hipError_t launch_tl2_stream(const FusedLinears& L, const float* x, int K, int8_t* xq, float* x_scale,
                             int32_t* x_rowsum, hipStream_t stream, bool lossy = false);

// ELUT for integer weights of other cardinalities: formats c4g2, c5g2 and c3g5 (table lookups, up to 4 tokens per
// launch for the 2-weight groups and 2 for c3g5; the launcher slices M).  Every weight of L in one launch.  With x
// (fp32, one token) the launch quantises the row itself and writes xq_out, s_out and rs_out as the quantiser would;
// otherwise it reads xq and x_scale (M tokens).
constexpr int kElutC4G2 = 0;
constexpr int kElutC5G2 = 1;
constexpr int kElutC3G5 = 2;
hipError_t launch_elut_generic(int fmt, const FusedLinears& L, const float* x, const int8_t* xq,
                               const float* x_scale, int M, int K, int8_t* xq_out, float* s_out, int32_t* rs_out,
                               hipStream_t stream);
hipError_t launch_pack_elut(int fmt, const int8_t* Wq, int N, int K, void* packed, hipStream_t stream);


}  // namespace bitnet
