// Decode GEMV for the I2_S layout (M <= 16 tokens): ternary x int8 accumulation (Eq. 1) on int8 MFMA,
// with the dequantisation epilogue fused.
//
// Weights are HBM-bound: each packed byte is read exactly once, with 16-byte non-temporal loads, one
// contiguous KiB per wave per 256-k block.  A 32-bit word of lane (r, q) holds 16 codes c = t + 1 of
// row r; shifting by 2f and masking 0x03030303 gives the four int8 codes of k = 4f .. 4f+3, which is
// exactly the byte order of the matching activation word.  So the unpacked word feeds the B operand of
// v_mfma_i32_16x16x64_i8 directly (B column = weight row, A row = token; rows past the tokens repeat a
// real token and are not stored).  The codes carry a +1 offset, removed by subtracting sum_k xq[m, k]:
// read from x_rowsum (written by the quantiser) when given, otherwise taken with a second MFMA against an
// all-ones B over the same k.
//
// Every weight load of a batch is issued before the first of them is used, as one unconditional 16-byte
// load per lane; a conditional load shape (the short last block) would make the compiler wait for each load
// before issuing the next.  One launch may cover several weights that share the activation (the row groups
// of the weights are concatenated).  No work group depends on another, so no device-wide fence is needed (an
// agent-scope release writes back the whole L2 of the XCD, which costs more than these GEMVs).
//
// i2s_decode_kernel (tokens already quantised): one work group per 16-row group holding the whole K; its 4,
// 8 or 16 waves take every WAVES-th 256-k block and reduce through LDS.
//
// i2s_gemv1_stream_kernel (one token, quantiser fused, Sec. 2.1): each work group quantises the fp32 row
// once into LDS codes and then streams row groups, keeping the next batch of weight loads in flight while it
// multiplies the current one.
#include "bitnet_internal.hpp"

#include <type_traits>

namespace bitnet {
namespace {

// Words per lane of block kb: 4 for a full 256-k block, (K mod 256) / 64 for a short last one.
__device__ __forceinline__ int block_T(int kb, int nfull, int Tlast) { return kb < nfull ? 4 : Tlast; }

// The 16 bytes that hold this lane's words of block kb.  A full block gives lane l the words at 16 l; a short
// block (T words per lane, 256 T bytes) gives them at 4 T l, and lanes near its end read a window moved back to
// end inside the block, so no lane reads past the row group.  The load is unconditional (the caller clamps kb
// to a real block), which keeps every weight load of a batch in flight together.
__device__ __forceinline__ v4u load_block(const uint8_t* wbase, int kb, int T, int lane) {
    const int want = 4 * T * lane;
    const int off = want < 256 * T - 16 ? want : 256 * T - 16;
    return load_stream16(wbase + (size_t)kb * 1024 + off);
}

// Word j of this lane's block after load_block: words are shifted by the window's move (0 for full blocks).
__device__ __forceinline__ uint32_t block_word(const v4u& w, int j, int T, int lane) {
    if (T == 4) return word_of(w, j);
    const int want = 4 * T * lane;
    const int sh = want < 256 * T - 16 ? 0 : (want - (256 * T - 16)) >> 2;
    const int i = j + sh;
    return i == 0 ? w.x : i == 1 ? w.y : i == 2 ? w.z : w.w;
}

template <int WAVES, int U, bool HAS_RS, int FMT>
__global__ __launch_bounds__(64 * WAVES) void i2s_decode_kernel(FusedLinears L, const int8_t* __restrict__ xq,
                                                                const float* __restrict__ x_scale,
                                                                const int32_t* __restrict__ x_rowsum, int M, int K) {
    __shared__ v4i red[WAVES][64];

    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int li, rg;
    locate(L, xcd_logical_id(blockIdx.x, gridDim.x), li, rg);
    const int N = pick(L.N, li);
    const int nkb = (K + kI2sBlockK - 1) / kI2sBlockK;
    const int nfull = K / kI2sBlockK;
    const int Tlast = nkb > nfull ? (K - nfull * kI2sBlockK) / kSubK : 4;
    const int q = lane >> 4, r = lane & 15;
    // A operand: row = token r, 16 k per lane group q.  Rows past M repeat token 0; their D rows are not stored.
    const int8_t* arow = xq + (size_t)(r < M ? r : 0) * K + 16 * q;
    const uint8_t* wbase = pick(L.packed, li) + (size_t)rg * 4 * K;
    const v4i zero = {0, 0, 0, 0};

    // epilogue operands first: their round trips overlap the weight stream
    const float beta = *pick(L.w_scale, li);
    float xs_m[4];
    int rs_m[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const int m = 4 * q + v;
        xs_m[v] = m < M ? x_scale[m] : 1.0f;
        rs_m[v] = (HAS_RS && m < M) ? x_rowsum[m] : 0;
    }

    v4i acc = zero, rowsum = zero;
    const v4i ones = {0x01010101, 0x01010101, 0x01010101, 0x01010101};
    for (int kb0 = wave; kb0 < nkb; kb0 += WAVES * U) {
        // the batch's weights, then its activation operands: all loads issued before the first MFMA
        v4u wv[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kb = min(kb0 + WAVES * u, nkb - 1);
            wv[u] = load_block(wbase, kb, block_T(kb, nfull, Tlast), lane);
        }
        v4i av[U][4];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kb = min(kb0 + WAVES * u, nkb - 1);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int k = min(kb * kI2sBlockK + kSubK * j, K - kSubK);   // past a short block: any real k
                av[u][j] = order_a<FMT>(*reinterpret_cast<const v4i*>(arow + k));
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kb = kb0 + WAVES * u;
            if (kb < nkb) {
                const int T = block_T(kb, nfull, Tlast);
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    if (j < T) {
                        acc = mfma16x16x64(av[u][j], decode_b<FMT>(block_word(wv[u], j, T, lane)), acc);
                        if (!HAS_RS) rowsum = mfma16x16x64(av[u][j], ones, rowsum);
                    }
                }
            }
        }
    }

    red[wave][lane] = acc - rowsum;
    __syncthreads();
    if (wave != 0) return;
    acc = red[0][lane];
#pragma unroll
    for (int w = 1; w < WAVES; ++w) acc += red[w][lane];

    // Output element v of lane l is D[row 4*(l/16) + v][col l%16]: token m = 4q + v, weight row r.
    float* y = pick(L.y, li);
    int32_t* acc_out = pick(L.acc, li);
    const int n = rg * kRowsPerGroup + r;
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const int m = 4 * q + v;
        if (m < M) {
            const float sc = beta / xs_m[v];
            const int val = acc[v] - rs_m[v];
            y[(size_t)m * N + n] = (float)val * sc;
            if (acc_out) acc_out[(size_t)m * N + n] = val;
        }
    }
}

// Up to 16 tokens, already quantised, streaming (every wave's blocks of a row group fit one batch: K <= 256 U
// WAVES).  Each wave copies the codes of its own k-blocks, all tokens, into LDS once (rows of K + 16 bytes, so
// the 16 token rows of one MFMA operand fall in different banks); they are the MFMA A operands (row = token;
// rows past M repeat token 0 and are not stored) of every row group it multiplies, and no other wave reads
// them.  The work group then walks row groups as the single-token kernel does, two batches of weights in flight.
// HAS_ACC: some weight of the launch also stores its int32 sums (the parity hook); the other instance holds no
// code for them (2% of the eight-token step).
//
// Token slices (more than 16 tokens, the small-batch regime): blockIdx.y is a slice of `slice` tokens; every slice
// walks the same row groups in the same order, and with gridDim.x a multiple of 8 the work groups (x, y) of all
// slices run on the XCD x % 8, so the slices of a row group meet its weight bytes in one L2 rather than each
// fetching them from HBM.
template <int WAVES, int U, int MG, bool HAS_RS, bool HAS_ACC, int FMT>
__global__ __launch_bounds__(64 * WAVES) void i2s_decode_stream_kernel(FusedLinears L, const int8_t* __restrict__ xq,
                                                                       const float* __restrict__ x_scale,
                                                                       const int32_t* __restrict__ x_rowsum, int M,
                                                                       int K, int slice) {
    extern __shared__ __align__(16) int8_t xs[];      // M rows of K + 16 codes
    __shared__ v4i part[2][WAVES][64];
    __shared__ int tsum[WAVES][16];

    // this work group's token slice: tokens m0 .. m0 + M - 1
    const int m0 = (int)blockIdx.y * slice;
    M = min(M - m0, slice);
    xq += (size_t)m0 * K;
    x_scale += m0;
    if (HAS_RS) x_rowsum += m0;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int q = lane >> 4, r = lane & 15;
    const int G = gridDim.x, bid = blockIdx.x;
    const int nkb = (K + kI2sBlockK - 1) / kI2sBlockK;
    const int nfull = K / kI2sBlockK;
    const int Tlast = nkb > nfull ? (K - nfull * kI2sBlockK) / kSubK : 4;
    const int S = (L.total - bid + G - 1) / G;                // row groups of this work group, one batch each
    const int stride = K + 16;
    const uint32_t off_full = 16u * lane;
    const int want_tail = 4 * Tlast * lane;
    const uint32_t off_tail = (uint32_t)min(want_tail, 256 * Tlast - 16);
    const int sh_tail = (want_tail - (int)off_tail) >> 2;

    auto issue = [&](v4u (&w)[U], float& bw, int st) {
        int li, rg;
        locate(L, bid + st * G, li, rg);
        const uint8_t* wbase = pick(L.packed, li) + (size_t)rg * 4 * K;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kb = min(wave + WAVES * u, nkb - 1);
            w[u] = load_stream16(wbase + (size_t)kb * 1024 + (kb < nfull ? off_full : off_tail));
        }
        bw = *pick(L.w_scale, li);
    };

    // 1. this wave's blocks of every token, into LDS: one 16-byte chunk per lane, four token rows per load
    //    (loads clamped to real addresses, stores only where the chunk is real)
    constexpr int kMaxGroups = MG;                             // token groups of 4 (M <= 4 MG)
    v4i ast[U][kMaxGroups];
    const int c16 = lane & 15;
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
        for (int mg = 0; mg < kMaxGroups; ++mg) {
            const int m = min(4 * mg + (lane >> 4), M - 1);
            const int k = min((wave + WAVES * u) * kI2sBlockK + 16 * c16, K - 16);
            ast[u][mg] = *reinterpret_cast<const v4i*>(xq + (size_t)m * K + k);
        }
    // epilogue operands of tokens m = 4q + v
    float xs_m[4];
    int rs_m[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        const int m = 4 * q + v;
        xs_m[v] = m < M ? x_scale[m] : 1.0f;
        rs_m[v] = (HAS_RS && m < M) ? x_rowsum[m] : 0;
    }
    // the copy into LDS (after the first weight loads are issued) and, without x_rowsum, each token's code sum
    // over this wave's blocks: lanes of one row of 16 hold one token, reduced with DPP
    auto stage = [&]() {
        int tp[kMaxGroups];
#pragma unroll
        for (int mg = 0; mg < kMaxGroups; ++mg) tp[mg] = 0;
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int mg = 0; mg < kMaxGroups; ++mg) {
                const int m = 4 * mg + (lane >> 4);
                const int k = (wave + WAVES * u) * kI2sBlockK + 16 * c16;
                if (m < M && k < K) {
                    *reinterpret_cast<v4i*>(xs + m * stride + k) = order_a<FMT>(ast[u][mg]);
                    if (!HAS_RS) {
                        const v4i a4 = ast[u][mg];
                        tp[mg] = byte_sum4((uint32_t)a4.x, byte_sum4((uint32_t)a4.y,
                                                                    byte_sum4((uint32_t)a4.z,
                                                                              byte_sum4((uint32_t)a4.w, tp[mg]))));
                    }
                }
            }
        if (!HAS_RS) {
#pragma unroll
            for (int mg = 0; mg < kMaxGroups; ++mg) {
                int t = tp[mg];
#pragma unroll
                for (int i = 0; i < 4; ++i) t += dpp_row_step(t, i);      // sum over the 16 lanes of the row
                if (c16 == 0 && 4 * mg + (lane >> 4) < 16) tsum[wave][4 * mg + (lane >> 4)] = t;
            }
        }
        // the codes a lane wrote are MFMA operands of other lanes of this wave (tsum is read after a barrier)
        wave_lds_handoff();
    };

    const v4i zero = {0, 0, 0, 0};
    const int8_t* arow = xs + (r < M ? r : 0) * stride + 16 * q;
    int par = 0;
    bool rs_ready = HAS_RS;
    auto compute = [&](const v4u (&w)[U], float bw, int st) {
        v4i acc = zero;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kb = wave + WAVES * u;
            const int8_t* ab = arow + kb * kI2sBlockK;
            if (kb < nfull) {
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc = mfma16x16x64(*reinterpret_cast<const v4i*>(ab + kSubK * j), decode_b<FMT>(word_of(w[u], j)),
                                       acc);
            } else if (kb < nkb) {
#pragma unroll
                for (int j = 0; j < 3; ++j) {
                    if (j < Tlast) {
                        const int i = j + sh_tail;
                        const uint32_t wd = i == 0 ? w[u].x : i == 1 ? w[u].y : i == 2 ? w[u].z : w[u].w;
                        acc = mfma16x16x64(*reinterpret_cast<const v4i*>(ab + kSubK * j), decode_b<FMT>(wd), acc);
                    }
                }
            }
        }
        part[par][wave][lane] = acc;
        __syncthreads();
        if (!rs_ready) {                 // past a barrier: the waves' code sums are in LDS
            rs_ready = true;
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                int t = 0;
                for (int w2 = 0; w2 < WAVES; ++w2) t += tsum[w2][(4 * q + v) & 15];
                rs_m[v] = t;
            }
        }
        if (wave == 0 && 4 * q < M) {
            v4i tot = part[par][0][lane];
#pragma unroll 4
            for (int w2 = 1; w2 < WAVES; ++w2) tot += part[par][w2][lane];
            int li, rg;
            locate(L, bid + st * G, li, rg);
            const int N = pick(L.N, li);
            const int n = rg * kRowsPerGroup + r;
            float* y = pick(L.y, li);
            int32_t* acc_out = pick(L.acc, li);
            // D element v of lane l is row 4 (l / 16) + v (token), column l % 16 (weight row)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int m = 4 * q + v;
                if (m < M) {
                    const int val = tot[v] - rs_m[v];
                    y[(size_t)(m0 + m) * N + n] = (float)val * (bw / xs_m[v]);
                    if constexpr (HAS_ACC) {
                        if (acc_out) acc_out[(size_t)(m0 + m) * N + n] = val;
                    }
                }
            }
        }
        par ^= 1;
    };

    // Steps are instantiated for one and for several row groups per work group, so that no two paths with
    // different loads in flight join.
    auto run = [&](auto depth) {
        constexpr int kDepth = decltype(depth)::value;
        v4u wa[U], wb[U];
        float ba = 0.0f, bb = 0.0f;
        // every wave's code loads enter the memory pipeline before any weight load (else the last waves' codes
        // queue behind the first waves' weight batches)
        __builtin_amdgcn_s_barrier();
        issue(wa, ba, 0);
        if constexpr (kDepth == 1) {
            stage();
            compute(wa, ba, 0);
        } else {
            issue(wb, bb, 1);
            stage();
            int st = 0;
            for (; st + 3 < S; st += 2) {
                compute(wa, ba, st);
                issue(wa, ba, st + 2);
                compute(wb, bb, st + 1);
                issue(wb, bb, st + 3);
            }
            if (st + 2 < S) {
                compute(wa, ba, st);
                issue(wa, ba, st + 2);
                compute(wb, bb, st + 1);
                compute(wa, ba, st + 2);
            } else {
                compute(wa, ba, st);
                compute(wb, bb, st + 1);
            }
        }
    };
    if (S == 1) run(std::integral_constant<int, 1>{});
    else run(std::integral_constant<int, 2>{});
}

// One token, streaming: each work group quantises the activation row once (Sec. 2.1), keeps its codes in LDS and
// then walks the row groups g = blockIdx.x, blockIdx.x + gridDim.x, ... of the launch, one batch of WAVES * U
// blocks at a time (a row group takes ceil(K / (256 WAVES U)) batches).  One batch is in flight while the row is
// quantised; after that two register sets of weight words alternate: the loads of the next batch are issued before
// the current one is multiplied, so the weight stream never waits for the arithmetic.  The last batch of a row group reduces the waves' partial sums through LDS
// (double-buffered, one barrier) and applies the epilogue.  Every A row holds the token's codes (LDS broadcast
// reads, no lane masking); D row 0 is the one stored.  AREG (one batch per row group): every step multiplies the
// same blocks of the wave, so their A operands are read from LDS once and kept in registers.
template <int WAVES, int U, int XV, int FMT, bool AREG>
__global__ __launch_bounds__(64 * WAVES) void i2s_gemv1_stream_kernel(FusedLinears L, const float* __restrict__ x,
                                                                      int K, int8_t* __restrict__ xq_out,
                                                                      float* __restrict__ s_out,
                                                                      int32_t* __restrict__ rs_out) {
    extern __shared__ __align__(16) int8_t xs[];      // the K codes of the token
    __shared__ int part[2][WAVES][16];
    __shared__ float redf[WAVES];
    __shared__ int redi[WAVES];
    constexpr int kPerBatch = WAVES * U;

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int q = lane >> 4, r = lane & 15;
    const int G = gridDim.x, bid = blockIdx.x;
    const int total = L.total;
    const int nkb = (K + kI2sBlockK - 1) / kI2sBlockK;
    const int nfull = K / kI2sBlockK;
    const int Tlast = nkb > nfull ? (K - nfull * kI2sBlockK) / kSubK : 4;
    const int nb = (nkb + kPerBatch - 1) / kPerBatch;        // batches per row group
    const int S = ((total - bid + G - 1) / G) * nb;           // this group's steps (the grid never exceeds total)
    // lane byte offsets within a block: full blocks, and the short last block's window (see load_block)
    const uint32_t off_full = 16u * lane;
    const int want_tail = 4 * Tlast * lane;
    const uint32_t off_tail = (uint32_t)min(want_tail, 256 * Tlast - 16);
    const int sh_tail = (want_tail - (int)off_tail) >> 2;

    // step s = batch s % nb of row group bid + (s / nb) G
    auto step_gb = [&](int st, int& g, int& b) {
        const int gi = nb == 1 ? st : st / nb;
        b = st - gi * nb;
        g = bid + gi * G;
    };
    // the loads of one step: the batch's weight words, then the weight's scale (loaded with every batch, so
    // the epilogue never waits on a load issued after it)
    auto issue = [&](v4u (&w)[U], float& bw, int st) {
        int g, b, li, rg;
        step_gb(st, g, b);
        locate(L, g, li, rg);
        const uint8_t* wbase = pick(L.packed, li) + (size_t)rg * 4 * K;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int kb = min(b * kPerBatch + wave + WAVES * u, nkb - 1);
            w[u] = load_stream16(wbase + (size_t)kb * 1024 + (kb < nfull ? off_full : off_tail));
        }
        bw = *pick(L.w_scale, li);
    };

    // The rest is instantiated twice, for work groups with one step and with several, so that neither path
    // joins the other: a join between paths with different numbers of loads in flight makes the compiler wait
    // for all of them.
    auto run = [&](auto multi) {
        constexpr bool kMulti = decltype(multi)::value;
        // 1. the activation row into registers, the first batch of weights, then the quantisation
        const float4* x4 = reinterpret_cast<const float4*>(x);
        const int K4 = K >> 2;
        float4 xv[XV];
    #pragma unroll
        for (int i = 0; i < XV; ++i) {
            const int e = tid + i * 64 * WAVES;
            const float4 v = x4[e < K4 ? e : K4 - 1];
            xv[i] = e < K4 ? v : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
        }
        // every wave's row loads enter the memory pipeline before any weight load: without this barrier the last
        // waves' row loads queue behind the first waves' weight batches, and the quantisation waits for them
        __builtin_amdgcn_s_barrier();
        // one batch in flight during the quantisation (step 0), the second (step 1) issued once the codes are made:
        // a second or third batch ahead of the quantisation delays the row's arrival more than it saves later
        v4u wa[U], wb[U];
        float ba = 0.0f, bb = 0.0f;
        issue(wa, ba, 0);
        __builtin_amdgcn_sched_barrier(0);   // keep the weight loads ahead of the quantisation arithmetic

        float amax = 0.0f;
    #pragma unroll
        for (int i = 0; i < XV; ++i)
            amax = fmaxf(amax, fmaxf(fmaxf(fabsf(xv[i].x), fabsf(xv[i].y)), fmaxf(fabsf(xv[i].z), fabsf(xv[i].w))));
        amax = wave_max_all(amax);
        if (lane == 0) redf[wave] = amax;
        __syncthreads();
        amax = redf[0];
    #pragma unroll
        for (int w = 1; w < WAVES; ++w) amax = fmaxf(amax, redf[w]);
        const float sx = 127.0f / fmaxf(amax, 1e-5f);
        int sum = 0;
    #pragma unroll
        for (int i = 0; i < XV; ++i) {
            const int e = tid + i * 64 * WAVES;
            if (e < K4) {
                const uint32_t c = quant4(xv[i], sx);
                sum = byte_sum4(c, sum);
                uint32_t cs = c;
                if constexpr (FMT == kFmtTl1) {
                    // the 16 codes of k = 16 (e / 4) .. + 15 in tl1_codes' order: word e % 4 of the group takes
                    // bytes of its own word and of its neighbour e ^ 1 (the next lane of the same quad)
                    const uint32_t nb = (uint32_t)dpp_row_step((int)c, 0);
                    cs = (e & 1) ? __builtin_amdgcn_perm(c, nb, 0x07050301u) : __builtin_amdgcn_perm(nb, c, 0x06040200u);
                }
                reinterpret_cast<uint32_t*>(xs)[e] = cs;
                if (bid == 0) reinterpret_cast<uint32_t*>(xq_out)[e] = c;
            }
        }
        // Codes 4e .. 4e+3 (e = tid + 64 WAVES i) lie in block e / 64, and e / 64 = wave (mod WAVES): every
        // wave quantised exactly the blocks it multiplies, so only the lanes of one wave exchange codes (an
        // LDS hand-off inside the wave, no work-group barrier).  The waves' code sums meet in the first
        // epilogue, which follows a barrier.
        if constexpr (kMulti) issue(wb, bb, 1);
        wave_lds_handoff();
        sum = wave_sum_all(sum);
        if (lane == 0) redi[wave] = sum;
        if (bid == 0 && tid == 0) s_out[0] = sx;
        int rowsum = 0;
        bool rowsum_ready = false;

        // 2. the stream
        const v4i zero = {0, 0, 0, 0};
        const int8_t* arow = xs + 16 * q;
        v4i areg[AREG ? U : 1][4];
        if constexpr (AREG) {
    #pragma unroll
            for (int u = 0; u < U; ++u)
    #pragma unroll
                for (int j = 0; j < 4; ++j) {
                    // k past a short block or past K: any real k (never multiplied)
                    const int k = min((wave + WAVES * u) * kI2sBlockK + kSubK * j, K - kSubK);
                    areg[u][j] = *reinterpret_cast<const v4i*>(arow + k);
                }
        }
        v4i acc = zero;
        int par = 0;
        auto compute = [&](const v4u (&w)[U], float bw, int st) {
            int g, b;
            step_gb(st, g, b);
            if (b == 0) acc = zero;
    #pragma unroll
            for (int u = 0; u < U; ++u) {
                const int kb = b * kPerBatch + wave + WAVES * u;
                const int8_t* ab = arow + kb * kI2sBlockK;
                if (kb < nfull) {
    #pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc = mfma16x16x64(AREG ? areg[AREG ? u : 0][j] : *reinterpret_cast<const v4i*>(ab + kSubK * j),
                                           decode_b<FMT>(word_of(w[u], j)), acc);
                } else if (kb < nkb) {
    #pragma unroll
                    for (int j = 0; j < 3; ++j) {
                        if (j < Tlast) {
                            const int i = j + sh_tail;
                            const uint32_t wd = i == 0 ? w[u].x : i == 1 ? w[u].y : i == 2 ? w[u].z : w[u].w;
                            acc = mfma16x16x64(AREG ? areg[AREG ? u : 0][j] : *reinterpret_cast<const v4i*>(ab + kSubK * j),
                                               decode_b<FMT>(wd), acc);
                        }
                    }
                }
            }
            if (b == nb - 1) {
                // token 0 is D row 0: element 0 of lanes 0..15
                if (q == 0) part[par][wave][r] = acc.x;
                __syncthreads();
                if (!rowsum_ready) {         // past a barrier: every wave's code sum is in LDS
                    rowsum_ready = true;
                    for (int w2 = 0; w2 < WAVES; ++w2) rowsum += redi[w2];
                    if (bid == 0 && tid == 0) rs_out[0] = rowsum;
                }
                if (wave == 0 && q == 0) {
                    int v = 0;
    #pragma unroll
                    for (int w2 = 0; w2 < WAVES; ++w2) v += part[par][w2][r];
                    int li, rg;
                    locate(L, g, li, rg);
                    const int n = rg * kRowsPerGroup + r;
                    const int val = v - rowsum;
                    pick(L.y, li)[n] = (float)val * (bw / sx);
                    int32_t* acc_out = pick(L.acc, li);
                    if (acc_out) acc_out[n] = val;
                }
                par ^= 1;
            }
        };
        // steps st and st + 1 are in flight; each register set is refilled right after it is multiplied.  The last
        // two or three steps are peeled so that no load is issued past the last step.
        if constexpr (!kMulti) {
            compute(wa, ba, 0);
            return;
        }
        int st = 0;
        for (; st + 3 < S; st += 2) {
            compute(wa, ba, st);
            issue(wa, ba, st + 2);
            compute(wb, bb, st + 1);
            issue(wb, bb, st + 3);
        }
        if (st + 2 < S) {
            compute(wa, ba, st);
            issue(wa, ba, st + 2);
            compute(wb, bb, st + 1);
            compute(wa, ba, st + 2);
        } else {
            compute(wa, ba, st);
            compute(wb, bb, st + 1);
        }
    };
    if (S == 1) run(std::false_type{});
    else run(std::true_type{});
}

template <int FMT, int WAVES, int U>
void launch_plain(const FusedLinears& L, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum, int M, int K,
                  hipStream_t stream) {
    const dim3 grid((unsigned)L.total), block(64 * WAVES);
    if (x_rowsum)
        hipLaunchKernelGGL((i2s_decode_kernel<WAVES, U, true, FMT>), grid, block, 0, stream, L, xq, x_scale, x_rowsum,
                           M, K);
    else
        hipLaunchKernelGGL((i2s_decode_kernel<WAVES, U, false, FMT>), grid, block, 0, stream, L, xq, x_scale, x_rowsum,
                           M, K);
}

template <int FMT, int WAVES>
void launch_plain_u(int U, const FusedLinears& L, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum,
                    int M, int K, hipStream_t stream) {
    if (U <= 1) launch_plain<FMT, WAVES, 1>(L, xq, x_scale, x_rowsum, M, K, stream);
    else if (U <= 2) launch_plain<FMT, WAVES, 2>(L, xq, x_scale, x_rowsum, M, K, stream);
    else launch_plain<FMT, WAVES, 4>(L, xq, x_scale, x_rowsum, M, K, stream);
}

constexpr int64_t kDecodeStageBytes = 128 * 1024;   // LDS for the tokens' codes in the multi-token stream

template <int FMT, int WAVES, int U, int XV, bool AREG = false>
hipError_t launch_stream(const FusedLinears& L, const float* x, int K, int8_t* xq, float* s, int32_t* rs,
                         hipStream_t stream) {
    auto kern = i2s_gemv1_stream_kernel<WAVES, U, XV, FMT, AREG>;
    const size_t lds = (size_t)K;
    // as many work groups as are resident at once, balanced so that every one walks the same number of row groups
    // (to within one).  16-wave groups: one per CU (a second resident group per CU, which the register use of the
    // one-batch start allows, measured slower on the 100B-class stack: 4.96 against 4.74 ms per step); 4-wave
    // groups: as many as fit, every row group in flight at once
    int occ = 1;
    if (WAVES < 16 &&
        (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, reinterpret_cast<const void*>(kern), 64 * WAVES, lds) !=
             hipSuccess ||
         occ <= 0))
        occ = 1;
    const int total = L.total;
    const int64_t max_g = (int64_t)device_cus() * occ;
    const int64_t rounds = (total + max_g - 1) / max_g;
    const int grid = (int)((total + rounds - 1) / rounds);
    hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(64 * WAVES), lds, stream, L, x, K, xq, s, rs);
    return hipGetLastError();
}

template <int FMT, int WAVES, int U>
hipError_t launch_stream_xv(const FusedLinears& L, const float* x, int K, int8_t* xq, float* s, int32_t* rs,
                            hipStream_t stream) {
    const int xv = (K / 4 + 64 * WAVES - 1) / (64 * WAVES);
    if constexpr (WAVES == 16 && U <= 3) {
        // one batch per row group: the A operands stay in registers (16 U of them; at U = 4 the kernel spills)
        if ((K + kI2sBlockK - 1) / kI2sBlockK <= WAVES * U) {
            if (xv <= 1) return launch_stream<FMT, WAVES, U, 1, true>(L, x, K, xq, s, rs, stream);
            if (xv <= 2) return launch_stream<FMT, WAVES, U, 2, true>(L, x, K, xq, s, rs, stream);
            if (xv <= 4) return launch_stream<FMT, WAVES, U, 4, true>(L, x, K, xq, s, rs, stream);
        }
    }
    if (xv <= 1) return launch_stream<FMT, WAVES, U, 1>(L, x, K, xq, s, rs, stream);
    if (xv <= 2) return launch_stream<FMT, WAVES, U, 2>(L, x, K, xq, s, rs, stream);
    if (WAVES < 8 || xv <= 4) return launch_stream<FMT, WAVES, U, 4>(L, x, K, xq, s, rs, stream);
    if (xv <= 8) return launch_stream<FMT, WAVES, U, 8>(L, x, K, xq, s, rs, stream);
    // rows just past 8 loads per thread (K = 33024: 9) load only what they need
    if (xv <= 9) return launch_stream<FMT, WAVES, U, 9>(L, x, K, xq, s, rs, stream);
    if (xv <= 12) return launch_stream<FMT, WAVES, U, 12>(L, x, K, xq, s, rs, stream);
    return launch_stream<FMT, WAVES, U, 16>(L, x, K, xq, s, rs, stream);
}

// M tokens in slices of `slice` (M <= slice: one slice, the whole launch on one token set).
template <int FMT, int W, int U, int MG>
hipError_t launch_mstream(const FusedLinears& L, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum,
                          int M, int K, hipStream_t stream, int slice = 16) {
    bool has_acc = false;
    for (int i = 0; i < L.count; ++i) has_acc = has_acc || L.acc[i] != nullptr;
    const void* kern = has_acc ? reinterpret_cast<const void*>(i2s_decode_stream_kernel<W, U, MG, true, true, FMT>)
                               : reinterpret_cast<const void*>(i2s_decode_stream_kernel<W, U, MG, true, false, FMT>);
    const int per = M < slice ? M : slice;                    // tokens of one slice
    const int slices = (M + per - 1) / per;
    const size_t lds = (size_t)per * (K + 16);
    int occ = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kern, 64 * W, lds) != hipSuccess || occ <= 0) occ = 1;
    int64_t max_g = (int64_t)device_cus() * occ;
    if (slices > 1) max_g = max_g / slices / kNumXcd * kNumXcd;  // every slice resident at once, XCD-aligned columns
    if (max_g < kNumXcd) max_g = kNumXcd;
    const int64_t rounds = (L.total + max_g - 1) / max_g;
    int64_t gx = (L.total + rounds - 1) / rounds;
    if (slices > 1 && gx > kNumXcd) gx = gx / kNumXcd * kNumXcd;
    const dim3 grid((unsigned)gx, (unsigned)slices), block(64 * W);
    if (has_acc)
        hipLaunchKernelGGL((i2s_decode_stream_kernel<W, U, MG, true, true, FMT>), grid, block, lds, stream, L, xq,
                           x_scale, x_rowsum, M, K, per);
    else
        hipLaunchKernelGGL((i2s_decode_stream_kernel<W, U, MG, true, false, FMT>), grid, block, lds, stream, L, xq,
                           x_scale, x_rowsum, M, K, per);
    return hipGetLastError();
}

template <int FMT, int W, int U>
hipError_t launch_mstream_m(const FusedLinears& L, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum,
                            int M, int K, hipStream_t stream, int slice) {
    const int per = M < slice ? M : slice;                    // tokens per work group
    if (per <= 4) return launch_mstream<FMT, W, U, 1>(L, xq, x_scale, x_rowsum, M, K, stream, slice);
    if (per <= 8) return launch_mstream<FMT, W, U, 2>(L, xq, x_scale, x_rowsum, M, K, stream, slice);
    if (per <= 12) return launch_mstream<FMT, W, U, 3>(L, xq, x_scale, x_rowsum, M, K, stream, slice);
    return launch_mstream<FMT, W, U, 4>(L, xq, x_scale, x_rowsum, M, K, stream, slice);
}

}  // namespace

// Compute units of the current device (cached per device).
int device_cus() {
    static int cus[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (cus[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
        cus[dev] = n;
    }
    return cus[dev];
}

// Waves per work group and blocks per wave per batch.  All waves of a launch should be resident at once
// (about 4096 on 256 CUs at the register use of these kernels): take the widest group (16, 8 or 4 waves) that
// keeps the launch within that, and let each wave load all of its blocks in one batch where the register
// budget allows (max_u).
void decode_shape(int64_t groups, int64_t K, int max_u, int min_waves, int& waves, int& u) {
    const int nkb = (int)((K + kI2sBlockK - 1) / kI2sBlockK);
    waves = 4;
    if (groups * 16 <= 4096) waves = 16;
    else if (groups * 8 <= 4096) waves = 8;
    if (waves < min_waves) waves = min_waves;
    while (waves < 16 && (nkb + waves - 1) / waves > max_u) waves *= 2;   // long K: one batch per wave
    u = (nkb + waves - 1) / waves;
    if (u > max_u) u = max_u;
}

template <int FMT>
hipError_t launch_decode_fmt(const FusedLinears& L, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum,
                             int M, int K, hipStream_t stream) {
    const int nkb = (K + kI2sBlockK - 1) / kI2sBlockK;
    const int cus = device_cus();
    // tokens per work group: up to 16 (one MFMA's rows), as many as fit in LDS; more tokens run as token slices
    int slice = 16;
    while (slice > 4 && (int64_t)slice * (K + 16) > kDecodeStageBytes) slice -= 4;
    const int per = M < slice ? M : slice;
    const bool fits = (int64_t)per * (K + 16) <= kDecodeStageBytes;   // a slice's codes fit in LDS
    if (M > 16 && !(x_rowsum && fits && nkb <= 64)) return hipErrorInvalidValue;
    if (x_rowsum && fits && nkb <= 16 && L.total > cus / 2) {
        // 4-wave work groups (K <= 4096) where the launch has more row groups than half the CUs: each group stages
        // the codes once as the 16-wave groups do, without waiting on the slowest of 16 waves at each barrier
        const int u4 = (nkb + 3) / 4;
        if (u4 <= 1) return launch_mstream_m<FMT, 4, 1>(L, xq, x_scale, x_rowsum, M, K, stream, slice);
        if (u4 <= 2) return launch_mstream_m<FMT, 4, 2>(L, xq, x_scale, x_rowsum, M, K, stream, slice);
        if (u4 <= 3) return launch_mstream_m<FMT, 4, 3>(L, xq, x_scale, x_rowsum, M, K, stream, slice);
        return launch_mstream_m<FMT, 4, 4>(L, xq, x_scale, x_rowsum, M, K, stream, slice);
    }
    if (x_rowsum && fits && nkb <= 64) {
        // 16-wave work groups, all of a row group's blocks in one batch; past what fits on the chip they stream
        const int u16 = (nkb + 15) / 16;
        if (u16 <= 1) return launch_mstream_m<FMT, 16, 1>(L, xq, x_scale, x_rowsum, M, K, stream, slice);
        if (u16 <= 2) return launch_mstream_m<FMT, 16, 2>(L, xq, x_scale, x_rowsum, M, K, stream, slice);
        if (u16 <= 3) return launch_mstream_m<FMT, 16, 3>(L, xq, x_scale, x_rowsum, M, K, stream, slice);
        return launch_mstream_m<FMT, 16, 4>(L, xq, x_scale, x_rowsum, M, K, stream, slice);
    }
    int waves, u;
    decode_shape(L.total, K, 4, 4, waves, u);
    switch (waves) {
        case 4: launch_plain_u<FMT, 4>(u, L, xq, x_scale, x_rowsum, M, K, stream); break;
        case 8: launch_plain_u<FMT, 8>(u, L, xq, x_scale, x_rowsum, M, K, stream); break;
        default: launch_plain_u<FMT, 16>(u, L, xq, x_scale, x_rowsum, M, K, stream); break;
    }
    return hipGetLastError();
}

template <int FMT>
hipError_t launch_gemv1_fmt(const FusedLinears& L, const float* x, int K, int8_t* xq, float* x_scale,
                            int32_t* x_rowsum, hipStream_t stream) {
    const int nkb = (K + kI2sBlockK - 1) / kI2sBlockK;
    const int cus = device_cus();
    if (L.total > cus / 2 && L.total <= 8 * cus && nkb <= 16) {
        // every row group in flight at once: one per 4-wave work group, from half a group per CU up to eight per
        // CU (a 16-wave group waits on its slowest wave at the quantisation and at the reduction)
        const int u = (nkb + 3) / 4;
        if (u <= 1) return launch_stream_xv<FMT, 4, 1>(L, x, K, xq, x_scale, x_rowsum, stream);
        if (u <= 2) return launch_stream_xv<FMT, 4, 2>(L, x, K, xq, x_scale, x_rowsum, stream);
        if (u <= 3) return launch_stream_xv<FMT, 4, 3>(L, x, K, xq, x_scale, x_rowsum, stream);
        return launch_stream_xv<FMT, 4, 4>(L, x, K, xq, x_scale, x_rowsum, stream);
    }
    if (L.total <= cus && nkb > 32 && K <= 32768) {
        // one row group per work group, long rows: 8-wave groups, so that a row group is at least two batches and
        // only the first is in flight while the row is quantised (the 8B-class down projection, 14336 -> 4096:
        // 16 waves 22.4 us per layer set, 8 waves 21.6 us)
        constexpr int kW8 = 8;
        const int nb8 = (nkb + 4 * kW8 - 1) / (4 * kW8);
        const int u8 = (nkb + kW8 * nb8 - 1) / (kW8 * nb8);
        if (u8 <= 3) return launch_stream_xv<FMT, kW8, 3>(L, x, K, xq, x_scale, x_rowsum, stream);
        return launch_stream_xv<FMT, kW8, 4>(L, x, K, xq, x_scale, x_rowsum, stream);
    }
    // 16-wave work groups, up to four 256-k blocks per wave per batch, the batches of a row group balanced;
    // past what fits on the chip at once the work groups stream
    constexpr int kWaves = 16;
    const int nb = (nkb + 4 * kWaves - 1) / (4 * kWaves);
    const int u = (nkb + kWaves * nb - 1) / (kWaves * nb);
    if (u <= 1) return launch_stream_xv<FMT, kWaves, 1>(L, x, K, xq, x_scale, x_rowsum, stream);
    if (u <= 2) return launch_stream_xv<FMT, kWaves, 2>(L, x, K, xq, x_scale, x_rowsum, stream);
    if (u <= 3) return launch_stream_xv<FMT, kWaves, 3>(L, x, K, xq, x_scale, x_rowsum, stream);
    return launch_stream_xv<FMT, kWaves, 4>(L, x, K, xq, x_scale, x_rowsum, stream);
}

hipError_t launch_i2s_decode(const FusedLinears& L, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum,
                             int M, int K, hipStream_t stream, int fmt) {
    return fmt == kFmtTl1 ? launch_decode_fmt<kFmtTl1>(L, xq, x_scale, x_rowsum, M, K, stream)
                          : launch_decode_fmt<kFmtI2s>(L, xq, x_scale, x_rowsum, M, K, stream);
}

hipError_t launch_i2s_gemv1_stream(const FusedLinears& L, const float* x, int K, int8_t* xq, float* x_scale,
                                   int32_t* x_rowsum, hipStream_t stream, int fmt) {
    return fmt == kFmtTl1 ? launch_gemv1_fmt<kFmtTl1>(L, x, K, xq, x_scale, x_rowsum, stream)
                          : launch_gemv1_fmt<kFmtI2s>(L, x, K, xq, x_scale, x_rowsum, stream);
}

}  // namespace bitnet
