// Prefill GEMM for the I2_S layout (M > 16 tokens): ternary x int8 accumulation (Eq. 1) as a dense int8
// contraction on v_mfma_i32_32x32x32_i8, with the dequantisation epilogue fused.  The paper leaves prefill
// open (Sec. "Limitations": prefill is compute-bound, so its CPU methods do not apply); this kernel is the
// MFMA-bound design for it.  (On gfx950 the 32x32x32 int8 MFMA sustains about twice the rate of the 16x16x64
// one, so the contraction uses the former.)
//
// Operand reuse decides this kernel: per output tile the int8 activations cost 1 byte per k per token row and
// the packed weights 1/4 byte per k per weight row, so tiles are wide along N (weights) to reuse each staged
// activation row many times.  A work group of WM x WN waves computes a 128-token x (128*WN)-row tile; each
// wave owns (128/WM) x 128 (MT x 4 MFMA tiles of 32 x 32, MT = 4/WM).  The widest tile uses one wave per SIMD
// with its 256 accumulator registers in AGPRs.  K advances in 256-k stages, the I2_S block size, so the
// packed weights of one row group and stage are one contiguous KiB.  Lane (j, h) of a wave (j = lane % 32,
// h = lane / 32) needs, for its weight row j, the 16 codes of k-step s at k = 32 s + 16 h: word s/2 of the
// layout's lane chunk q = 2 (s % 2) + h; each lane loads those chunks straight into registers and unpacks them
// there, so the weights never pass through LDS.  The activation tile (128 x 256) is staged in LDS with rows
// padded to 272 bytes, double-buffered: one barrier per stage.  Activations are loaded into registers one
// stage ahead of their LDS store, the next stage's weight words at the start of each stage.  Tiles are
// ordered in groups of 4 token tiles so that the work groups resident on one XCD share activation and weight
// tiles in its L2.
//
// The codes are t + 1: sum_k xq[m, k] is subtracted in the epilogue, either from x_rowsum (written by the
// quantiser) or accumulated here by the threads that stage the activation rows.
#include "bitnet_internal.hpp"

namespace bitnet {
namespace {

typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kBM = 128, kBK = 256;
constexpr int kARow = kBK + 16;            // padded LDS row of the activation tile
constexpr int kGroupM = 4;                 // token tiles per scheduling group

__device__ __forceinline__ int byte_sum(const v4i& v) {
    const int ones = 0x01010101;
    int s = __builtin_amdgcn_sdot4(v.x, ones, 0, false);
    s = __builtin_amdgcn_sdot4(v.y, ones, s, false);
    s = __builtin_amdgcn_sdot4(v.z, ones, s, false);
    return __builtin_amdgcn_sdot4(v.w, ones, s, false);
}

template <int WM, int WN, bool HAS_RS>
__global__ __launch_bounds__(64 * WM * WN) void i2s_prefill_kernel(
    const uint8_t* __restrict__ packed, const float* __restrict__ w_scale, const int8_t* __restrict__ xq,
    const float* __restrict__ x_scale, const int32_t* __restrict__ x_rowsum, int M, int N, int K,
    float* __restrict__ y, int32_t* __restrict__ acc_out, int splits, int32_t* __restrict__ part) {
    constexpr int kThreads = 64 * WM * WN;
    constexpr int kBN = 128 * WN;
    constexpr int MT = 4 / WM;                               // 32-row MFMA tiles per wave along M
    constexpr int kChunks = kBM * (kBK / 16) / kThreads;     // 16-byte activation chunks per thread per stage
    __shared__ __align__(16) int8_t As[2][kBM * kARow];       // double-buffered activation tile
    __shared__ int rowsum_s[kBM];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave % WM, wn = wave / WM;
    const int j32 = lane & 31, h = lane >> 5;
    const int tiles_m = (M + kBM - 1) / kBM;
    const int tiles_n = (N + kBN - 1) / kBN;
    // split-K: the launch is splits slices of tiles; slice `split` takes stages [kb_lo, kb_hi)
    const int ntiles = gridDim.x / splits;
    const int split = blockIdx.x / ntiles;
    const int L = xcd_logical_id(blockIdx.x - split * ntiles, ntiles);
    // grouped order: kGroupM token tiles x all weight tiles per group, token tile fastest
    const int gsize = kGroupM * tiles_n;
    const int g = L / gsize, gl = L - g * gsize;
    const int gm = (tiles_m - g * kGroupM) < kGroupM ? (tiles_m - g * kGroupM) : kGroupM;
    const int tm = g * kGroupM + gl % gm, tn = gl / gm;
    const int m0 = tm * kBM, n0 = tn * kBN;
    const int nkb = (K + kBK - 1) / kBK;
    const int nfull = K / kBK;
    const int per_split = (nkb + splits - 1) / splits;
    const int kb_lo = split * per_split;
    const int kb_hi = min(nkb, kb_lo + per_split);
    const int nrg = N / kRowsPerGroup;
    const size_t rg_bytes = (size_t)4 * K;

    // weight row group and lane chunk of each 32-row tile of this wave
    int rg[4];
    bool rg_ok[4];
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) {
        rg[ni] = n0 / kRowsPerGroup + 8 * wn + 2 * ni + (j32 >> 4);
        rg_ok[ni] = rg[ni] < nrg;
    }
    const int r16 = j32 & 15;
    // Loads are unconditional (a conditional load shape makes the compiler wait for every load before the next):
    // rows past N load a real row group (never stored), and the short last block (Tl 64-k sub-tiles) is read
    // through a 16-byte window moved back to end inside it, its words shifted into place at use.
    const int Tl = nkb > nfull ? (K - nfull * kBK) / kSubK : 4;
    uint32_t rgoff[4];                                              // byte offset of the (clamped) row group
#pragma unroll
    for (int ni = 0; ni < 4; ++ni) rgoff[ni] = (uint32_t)(rg[ni] < nrg ? rg[ni] : nrg - 1) * (uint32_t)rg_bytes;
    uint32_t offb_full[2], offb_tail[2];
    int shb_tail[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
        const int ql = 16 * (2 * c + h) + r16;                     // lane of the layout's chunk
        const int want = 4 * Tl * ql;
        offb_full[c] = 16u * ql;
        offb_tail[c] = (uint32_t)min(want, 256 * Tl - 16);
        shb_tail[c] = (want - (int)offb_tail[c]) >> 2;
    }

    const v4i zero4 = {0, 0, 0, 0};
    v16i acc[MT][4];
#pragma unroll
    for (int mi = 0; mi < MT; ++mi)
#pragma unroll
        for (int ni = 0; ni < 4; ++ni) acc[mi][ni] = v16i{};
    int rs[kChunks];
#pragma unroll
    for (int i = 0; i < kChunks; ++i) rs[i] = 0;

    v4i a_reg[kChunks];
    v4u bw0[4][2], bw1[4][2];          // weight words of even / odd stages: [tile][chunk: q = h, q = 2 + h]

    auto stage_T = [&](int kb) { return kb < nfull ? 4 : (K - nfull * kBK) / kSubK; };   // 64-k sub-tiles
    // 32-bit offsets from uniform bases (the library limits M K and N K / 4 below 2^32)
    auto load_a = [&](int kb) {
#pragma unroll
        for (int i = 0; i < kChunks; ++i) {
            const int c = tid + i * kThreads;
            const uint32_t row = (uint32_t)min(m0 + (c >> 4), M - 1);
            const uint32_t col = (uint32_t)min(kb * kBK + (c & 15) * 16, K - 16);
            a_reg[i] = *reinterpret_cast<const v4i*>(xq + (row * (uint32_t)K + col));
        }
    };
    auto load_b = [&](int kb, v4u (&dst)[4][2]) {
        const bool full = kb < nfull;
        const uint8_t* pk = packed + (size_t)kb * 1024;
#pragma unroll
        for (int ni = 0; ni < 4; ++ni)
#pragma unroll
            for (int c = 0; c < 2; ++c)
                dst[ni][c] = __builtin_nontemporal_load(
                    reinterpret_cast<const v4u*>(pk + (rgoff[ni] + (full ? offb_full[c] : offb_tail[c]))));
    };
    // Columns past K are stored as zeros: a short last stage then runs as a full one, the weight words past its
    // end (whatever the shifted window holds) meeting zero activations.
    auto store_a = [&](int buf, int kb) {
        const int kcols = kb < nfull ? kBK : kb < nkb ? 64 * Tl : 0;   // past the last stage: nothing counts
#pragma unroll
        for (int i = 0; i < kChunks; ++i) {
            const int c = tid + i * kThreads;
            const bool col_on = (c & 15) * 16 < kcols;
            const v4i a = col_on ? a_reg[i] : zero4;
            *reinterpret_cast<v4i*>(As[buf] + (c >> 4) * kARow + (c & 15) * 16) = a;
            if (!HAS_RS) rs[i] += (m0 + (c >> 4) < M) ? byte_sum(a) : 0;
        }
    };
    // the MFMAs of one stage: 8 steps of 32 k
    auto mac_stage = [&](int buf, const v4u (&b_cur)[4][2]) {
#pragma unroll
        for (int s = 0; s < 8; ++s) {
            v4i a[MT];
#pragma unroll
            for (int mi = 0; mi < MT; ++mi)
                a[mi] = *reinterpret_cast<const v4i*>(As[buf] + (32 * MT * wm + 32 * mi + j32) * kARow + 32 * s + 16 * h);
#pragma unroll
            for (int ni = 0; ni < 4; ++ni) {
                const v4i b = unpack_codes(word_of(b_cur[ni][s & 1], s >> 1));
#pragma unroll
                for (int mi = 0; mi < MT; ++mi)
                    acc[mi][ni] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[mi], b, acc[mi][ni], 0, 0, 0);
            }
        }
    };
    // the short last stage: move each chunk's words to the front (its load window was moved back)
    auto align_tail = [&](v4u (&b_cur)[4][2]) {
#pragma unroll
        for (int c = 0; c < 2; ++c) {
            const int sh = shb_tail[c];
#pragma unroll
            for (int ni = 0; ni < 4; ++ni) {
                const v4u w = b_cur[ni][c];
                v4u t;
                t.x = sh == 0 ? w.x : sh == 1 ? w.y : sh == 2 ? w.z : w.w;
                t.y = sh == 0 ? w.y : sh == 1 ? w.z : w.w;
                t.z = sh == 0 ? w.z : w.w;
                t.w = w.w;
                b_cur[ni][c] = t;
            }
        }
    };

    // Stage kb's activations are in LDS buffer kb % 2 and its weight words in bw0 / bw1 (even / odd).  Every
    // stage loads the next stage's weights at its start and, after its MFMAs, stores the next stage's
    // activations (loaded a stage earlier) and loads the ones after.  Indices past the last stage are clamped
    // to it: those loads repeat the last stage (cache hits) and nothing is computed from them.
    const int last = kb_hi - 1;
    load_a(kb_lo);
    load_b(kb_lo, bw0);
    store_a(0, kb_lo);
    load_a(min(kb_lo + 1, last));
    for (int kb = kb_lo; kb < kb_hi; kb += 2) {
        __syncthreads();                                  // stage kb is in As[0]; As[1] is free
        load_b(min(kb + 1, last), bw1);
        if (kb >= nfull) align_tail(bw0);
        mac_stage(0, bw0);
        store_a(1, kb + 1 < kb_hi ? kb + 1 : nkb);
        load_a(min(kb + 2, last));
        if (kb + 1 >= kb_hi) break;
        __syncthreads();                                  // stage kb + 1 is in As[1]; As[0] is free
        load_b(min(kb + 2, last), bw0);
        if (kb + 1 >= nfull) align_tail(bw1);
        mac_stage(1, bw1);
        store_a(0, kb + 2 < kb_hi ? kb + 2 : nkb);
        load_a(min(kb + 3, last));
    }

    if (part) {
        // split-K: this slice's exact partial sums (the code offset and the scales are applied when the
        // slices are summed)
        int32_t* pp = part + (size_t)split * M * N;
#pragma unroll
        for (int mi = 0; mi < MT; ++mi)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + 32 * MT * wm + 32 * mi + 8 * (v >> 2) + 4 * h + (v & 3);
                if (m >= M) continue;
#pragma unroll
                for (int ni = 0; ni < 4; ++ni)
                    if (rg_ok[ni]) pp[(size_t)m * N + rg[ni] * kRowsPerGroup + r16] = acc[mi][ni][v];
            }
        return;
    }

    if (HAS_RS) {
        if (tid < kBM) rowsum_s[tid] = (m0 + tid < M) ? x_rowsum[m0 + tid] : 0;
    } else {
        // the 16 threads of one row are 16 consecutive lanes
#pragma unroll
        for (int i = 0; i < kChunks; ++i) {
            int v = rs[i];
            v += __shfl_xor(v, 1, 64);
            v += __shfl_xor(v, 2, 64);
            v += __shfl_xor(v, 4, 64);
            v += __shfl_xor(v, 8, 64);
            const int c = tid + i * kThreads;
            if ((c & 15) == 0) rowsum_s[c >> 4] = v;
        }
    }
    __syncthreads();

    // D element v of lane (j, h): row 8 * (v / 4) + 4 * h + v % 4, column j.
    const float beta = *w_scale;
#pragma unroll
    for (int mi = 0; mi < MT; ++mi) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
            const int ml = 32 * MT * wm + 32 * mi + 8 * (v >> 2) + 4 * h + (v & 3);
            const int m = m0 + ml;
            if (m >= M) continue;
            const int rsum = rowsum_s[ml];
            const float sc = beta / x_scale[m];
#pragma unroll
            for (int ni = 0; ni < 4; ++ni) {
                if (!rg_ok[ni]) continue;
                const int n = rg[ni] * kRowsPerGroup + r16;
                const int val = acc[mi][ni][v] - rsum;
                y[(size_t)m * N + n] = (float)val * sc;
                if (acc_out) acc_out[(size_t)m * N + n] = val;
            }
        }
    }
}

// Sum of the split-K slices, then the epilogue: y = (sum - sum_k xq[m, k]) * (beta / s_m).  Four outputs of
// one row per thread.
__global__ __launch_bounds__(256) void prefill_splitk_finish(const int32_t* __restrict__ part, int splits, int M,
                                                             int N, const int32_t* __restrict__ x_rowsum,
                                                             const float* __restrict__ x_scale,
                                                             const float* __restrict__ w_scale, float* __restrict__ y,
                                                             int32_t* __restrict__ acc_out) {
    const int64_t i4 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;      // index of 4 outputs
    const int n4 = N >> 2;
    if (i4 >= (int64_t)M * n4) return;
    const int m = (int)(i4 / n4);
    const size_t off = (size_t)i4 * 4;
    v4i t = *reinterpret_cast<const v4i*>(part + off);
    for (int sp = 1; sp < splits; ++sp) t += *reinterpret_cast<const v4i*>(part + (size_t)sp * M * N + off);
    const int rs = x_rowsum[m];
    t -= (v4i){rs, rs, rs, rs};
    const float sc = *w_scale / x_scale[m];
    float4 o;
    o.x = (float)t.x * sc;
    o.y = (float)t.y * sc;
    o.z = (float)t.z * sc;
    o.w = (float)t.w * sc;
    *reinterpret_cast<float4*>(y + off) = o;
    if (acc_out) *reinterpret_cast<v4i*>(acc_out + off) = t;
}

template <int WM, int WN>
void launch_cfg(const uint8_t* pk, const float* w_scale, const int8_t* xq, const float* x_scale,
                const int32_t* x_rowsum, int M, int N, int K, float* y, int32_t* acc, int splits, int32_t* part,
                hipStream_t stream) {
    const unsigned tiles = (unsigned)(((M + kBM - 1) / kBM) * ((N + 128 * WN - 1) / (128 * WN)));
    const dim3 grid(tiles * (unsigned)splits), block(64 * WM * WN);
    if (x_rowsum)
        hipLaunchKernelGGL((i2s_prefill_kernel<WM, WN, true>), grid, block, 0, stream, pk, w_scale, xq, x_scale,
                           x_rowsum, M, N, K, y, acc, splits, part);
    else
        hipLaunchKernelGGL((i2s_prefill_kernel<WM, WN, false>), grid, block, 0, stream, pk, w_scale, xq, x_scale,
                           x_rowsum, M, N, K, y, acc, splits, part);
}

// Tile shape (the widest that still gives every CU some work) and split-K factor.  Splitting K keeps small
// grids busy: it aims at one work group per CU, with at least two 256-k stages per slice.
void prefill_plan(int64_t M, int64_t N, int64_t K, int& wn, int& splits) {
    const int64_t tiles_m = (M + kBM - 1) / kBM;
    int64_t tiles;
    if (tiles_m * ((N + 511) / 512) >= 192) {
        wn = 4;                                           // 128 x 512, 4 waves
        tiles = tiles_m * ((N + 511) / 512);
    } else if (tiles_m * ((N + 255) / 256) >= 96) {
        wn = 2;                                           // 128 x 256, 4 waves
        tiles = tiles_m * ((N + 255) / 256);
    } else {
        wn = 1;                                           // 128 x 128, 2 waves
        tiles = tiles_m * ((N + 127) / 128);
    }
    const int64_t nkb = (K + kBK - 1) / kBK;
    const int64_t cus = device_cus();
    // only grids that leave at least half the CUs idle: the slices' extra pass over M x N costs more elsewhere
    int64_t sp = 2 * tiles <= cus ? (cus + tiles - 1) / tiles : 1;
    if (sp > nkb / 2) sp = nkb / 2;
    if (sp > kMaxSplits) sp = kMaxSplits;
    splits = sp > 1 ? (int)sp : 1;
    // slices of whole stages: no empty slice
    if (splits > 1) {
        const int64_t per = (nkb + splits - 1) / splits;
        splits = (int)((nkb + per - 1) / per);
    }
}

}  // namespace

size_t prefill_workspace_bytes(int64_t M, int64_t N, int64_t K) {
    int wn, splits;
    prefill_plan(M, N, K, wn, splits);
    return splits > 1 ? (size_t)splits * (size_t)M * (size_t)N * sizeof(int32_t) : 0;
}

hipError_t launch_i2s_prefill(const void* packed, const float* w_scale, const int8_t* xq, const float* x_scale,
                              const int32_t* x_rowsum, int M, int N, int K, float* y, int32_t* acc, void* ws,
                              size_t ws_bytes, hipStream_t stream) {
    const uint8_t* pk = static_cast<const uint8_t*>(packed);
    int wn, splits;
    prefill_plan(M, N, K, wn, splits);
    // split-K needs the token sums and the workspace for the slices
    if (!x_rowsum || !ws || ws_bytes < (size_t)splits * M * N * sizeof(int32_t)) splits = 1;
    int32_t* part = splits > 1 ? static_cast<int32_t*>(ws) : nullptr;
    switch (wn) {
        case 4: launch_cfg<1, 4>(pk, w_scale, xq, x_scale, x_rowsum, M, N, K, y, acc, splits, part, stream); break;
        case 2: launch_cfg<2, 2>(pk, w_scale, xq, x_scale, x_rowsum, M, N, K, y, acc, splits, part, stream); break;
        default: launch_cfg<2, 1>(pk, w_scale, xq, x_scale, x_rowsum, M, N, K, y, acc, splits, part, stream); break;
    }
    if (splits > 1) {
        const int64_t n4 = (int64_t)M * (N / 4);
        hipLaunchKernelGGL(prefill_splitk_finish, dim3((unsigned)((n4 + 255) / 256)), dim3(256), 0, stream, part,
                           splits, M, N, x_rowsum, x_scale, w_scale, y, acc);
    }
    return hipGetLastError();
}

}  // namespace bitnet
