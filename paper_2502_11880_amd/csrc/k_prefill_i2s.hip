// Prefill GEMM for the I2_S layout (M > 16 tokens): ternary x int8 accumulation (Eq. 1) as a dense int8
// contraction on v_mfma_i32_32x32x32_i8, with the dequantisation epilogue fused.  The paper leaves prefill
// open (Sec. "Limitations": prefill is compute-bound, so its CPU methods do not apply); this kernel is the
// MFMA-bound design for it.  (On gfx950 the 32x32x32 int8 MFMA sustains about twice the rate of the 16x16x64
// one, so the contraction uses the former.)
//
// Work decomposition.  A work group of 8 waves computes a 128-token x (128 WN)-row output tile.  Each wave owns
// 64 tokens x 128 rows (2 x 4 MFMA tiles of 32 x 32, 128 accumulator registers), so two waves share every
// SIMD: while one waits on LDS or on the barrier, the other keeps the matrix core busy.  With WN = 4 the waves
// tile the 128 x 512 output 2 x 4; with WN = 2 they tile a 128 x 256 output 2 x 2 and each pair splits the k-steps
// of every stage (WK = 2 K-groups), the two partial tiles summed through LDS at the end: the narrower tile doubles
// the grid of small problems without exact partial sums going through HBM.  K advances in 256-k stages, the I2_S
// block size, so the packed weights of one row group and stage are one contiguous KiB.
//
// Operands.  Both are staged in LDS, double-buffered, one barrier per stage.  Every thread loads its 16-byte
// chunks of the next-but-one stage into registers (plain coalesced loads: a wave reads whole KiB runs) and
// writes them to LDS during the next stage's MFMAs, so a load has a whole stage to arrive and the copies
// overlap the matrix work.
//   * Activations: token rows padded to 272 bytes, so an MFMA operand read (32 rows, one 16-byte chunk each)
//     hits every bank once.
//   * Weights: stored as ready-made MFMA B operands.  Lane (j, h) of a wave (j = lane % 32, h = lane / 32)
//     needs, for its weight row j, the 16 codes of k-step s at k = 32 s + 16 h, i.e. word s / 2 of the layout's
//     lane chunk q = 2 (s % 2) + h.  The staging threads write each 16-byte layout chunk to the slot of the lane
//     that uses it, so a wave reads its 8 chunks of a stage with 8 contiguous 1 KiB LDS reads and unpacks the
//     2-bit codes in registers.  (Loaded straight into registers instead, every weight word would be fetched
//     by both token halves of the work group and would need a second register set.)
// (Direct global-to-LDS copies were measured too: the address unit handles them lane by lane, about 25 times
// the cache accesses of these loads, and the kernel ran at half the speed.)  Tiles are ordered in groups of 4
// token tiles so that the work groups resident on one XCD share activation and weight tiles in its L2.
//
// The codes are t + 1: sum_k xq[m, k] is subtracted in the epilogue, either from x_rowsum (written by the
// quantiser) or summed here from the activation operands.  The epilogue goes through LDS in two passes of 64
// token rows, so every wave stores 1 KiB runs of one output row (16 bytes per lane, streaming hint) instead of
// 128-byte pieces of two rows per scalar store.
#include "bitnet_internal.hpp"

namespace bitnet {
namespace {

typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int kBK = 256;                   // k per stage (one I2_S block)
constexpr int kGroupM = 4;                 // token tiles per scheduling group
constexpr int kBM = 128;                   // tokens per work group tile
constexpr int kWaves = 8, kThreads = 64 * kWaves;
constexpr int kARow = kBK + 16;            // padded LDS row of the activation tile
constexpr int kAChunks = kBM * (kBK / 16) / kThreads;         // 16-byte activation chunks per thread per stage

__device__ __forceinline__ int byte_sum(const v4i& v, int acc) {
    const int ones = 0x01010101;
    acc = __builtin_amdgcn_sdot4(v.x, ones, acc, false);
    acc = __builtin_amdgcn_sdot4(v.y, ones, acc, false);
    acc = __builtin_amdgcn_sdot4(v.z, ones, acc, false);
    return __builtin_amdgcn_sdot4(v.w, ones, acc, false);
}

// The weights of one launch: each owns a run of weight tiles (tile_start), its own rows, beta and outputs, and
// its slice of a split-K partial buffer (part_off; a slice holds M x sum N).
struct PrefillLinears {
    const uint8_t* packed[kMaxFused];
    const float* w_scale[kMaxFused];
    float* y[kMaxFused];
    int32_t* acc[kMaxFused];
    long long part_off[kMaxFused];
    int N[kMaxFused];
    int tile_start[kMaxFused + 1];   // first weight tile of each linear; INT_MAX past the last
    int tile_start_lo[kMaxFused];     // the same, 0 past the last (the value subtracted)
    int tiles_n;                      // weight tiles of the launch
    long long n_total;                // sum of N
};

template <typename T>
__device__ __forceinline__ T pick_linear(const T (&a)[kMaxFused], int li) {
    T v = a[0];
#pragma unroll
    for (int i = 1; i < kMaxFused; ++i) v = li == i ? a[i] : v;
    return v;
}

// HAS_ACC: some weight of the launch also stores its int32 sums (the parity hook); without it the epilogue holds
// no code for them (2% of the 2048-token step).
template <int WN, bool HAS_RS, bool HAS_ACC>
__global__ __attribute__((amdgpu_waves_per_eu(2, 2))) __launch_bounds__(kThreads) void i2s_prefill_kernel(
    PrefillLinears P, const int8_t* __restrict__ xq, const float* __restrict__ x_scale,
    const int32_t* __restrict__ x_rowsum, int M, int K, int splits, int32_t* __restrict__ part_all) {
    constexpr int MT = 2, NT = 4;                                 // 32 x 32 MFMA tiles per wave
    constexpr int WK = 4 / WN;                                    // K-groups: waves sharing one output tile
    constexpr int kBN = 128 * WN;
    constexpr int kSteps = 8 / WK;                                // 32-k steps per stage of each wave
    constexpr int kWPer = WN;                                     // 16-byte weight chunks per thread per stage
    constexpr int kAsBytes = 2 * kBM * kARow;
    constexpr int kWsBytes = 2 * WN * 8 * 64 * 16;
    constexpr int kRedBytes = (WK - 1) * 2 * WN * 64 * 128 * 4;   // partial tiles of the K-groups past the first
    constexpr int kSmem = (kAsBytes + kWsBytes) > kRedBytes ? (kAsBytes + kWsBytes) : kRedBytes;
    __shared__ __align__(16) int8_t smem[kSmem];
    __shared__ int rowsum_s[WK][kBM];
    int8_t (*As)[kBM * kARow] = reinterpret_cast<int8_t (*)[kBM * kARow]>(smem);
    v4u (*Ws)[WN * 8 * 64] = reinterpret_cast<v4u (*)[WN * 8 * 64]>(smem + kAsBytes);   // [column][step][lane]

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wm = wave & 1, wn = (wave >> 1) % WN, wk = (wave >> 1) / WN;
    const int j32 = lane & 31, h = lane >> 5;
    const int tiles_m = (M + kBM - 1) / kBM;
    const int tiles_n = P.tiles_n;
    // split-K: the launch is `splits` slices of tiles; slice `split` takes stages [kb_lo, kb_hi)
    const int ntiles = gridDim.x / splits;
    const int split = blockIdx.x / ntiles;
    const int L = xcd_logical_id(blockIdx.x - split * ntiles, ntiles);
    // grouped order: kGroupM token tiles x all weight tiles per group, token tile fastest
    const int gsize = kGroupM * tiles_n;
    const int g = L / gsize, gl = L - g * gsize;
    const int gm = (tiles_m - g * kGroupM) < kGroupM ? (tiles_m - g * kGroupM) : kGroupM;
    const int tm = g * kGroupM + gl % gm, tn_all = gl / gm;
    // the weight this tile belongs to (uniform: a scalar compare chain over the fixed maximum)
    int li = 0;
#pragma unroll
    for (int i = 1; i < kMaxFused; ++i) li = tn_all >= P.tile_start[i] ? i : li;
    const int tn = tn_all - pick_linear(P.tile_start_lo, li);
    const int N = pick_linear(P.N, li);
    const uint8_t* __restrict__ packed = pick_linear(P.packed, li);
    const float* __restrict__ w_scale = pick_linear(P.w_scale, li);
    float* __restrict__ y = pick_linear(P.y, li);
    int32_t* __restrict__ acc_out = pick_linear(P.acc, li);
    int32_t* __restrict__ part = part_all ? part_all + pick_linear(P.part_off, li) : nullptr;
    const int m0 = tm * kBM, n0 = tn * kBN;
    const int nkb = (K + kBK - 1) / kBK;
    const int nfull = K / kBK;
    const int per_split = (nkb + splits - 1) / splits;
    const int kb_lo = split * per_split;
    const int kb_hi = min(nkb, kb_lo + per_split);
    const int nrg = N / kRowsPerGroup;
    const int rg0 = n0 / kRowsPerGroup;

    // ---- activations: chunk c of a stage is token row c / 16, bytes 16 (c % 16) ----
    // Rows past M repeat row M - 1 (never stored); columns past K read a real column (they meet zero weight codes).
    v4i a_reg[kAChunks];
    auto load_a1 = [&](int kb, int i) {
        const int c = tid + i * kThreads;
        const uint32_t row = (uint32_t)min(m0 + (c >> 4), M - 1);
        const uint32_t col = min((uint32_t)(kb * kBK + (c & 15) * 16), (uint32_t)K - 16u);
        a_reg[i] = *reinterpret_cast<const v4i*>(xq + (row * (uint32_t)K + col));
    };
    auto store_a1 = [&](int buf, int i) {
        const int c = tid + i * kThreads;
        *reinterpret_cast<v4i*>(As[buf] + (c >> 4) * kARow + (c & 15) * 16) = a_reg[i];
    };
    auto store_a = [&](int buf) {
#pragma unroll
        for (int i = 0; i < kAChunks; ++i) store_a1(buf, i);
    };
    auto load_a = [&](int kb) {
#pragma unroll
        for (int i = 0; i < kAChunks; ++i) load_a1(kb, i);
    };

    // ---- weights, staged as per-step B operands ----
    // LDS record (wave column wn, step s, lane L) holds the four 4-byte words lane L of the waves in column wn needs
    // at k-step s, one per 32-row tile ni: word s / 2 of layout lane chunk q = 2 (s % 2) + L / 32, row 16 ((L / 16) % 2)
    // + L % 16 of row group 8 wn + 2 ni + (L / 16) % 2.  Thread t stages the records of (wn, s % 2, L) = (t / 128,
    // (t / 64) % 2, t % 64) for all four s of that parity: it loads the four 16-byte layout chunks of that lane chunk
    // (one per tile; a wave's loads cover two contiguous 512-byte runs each), transposes the words in registers and
    // writes four 16-byte records.  A full block gives lane chunk l 16 bytes at 16 l.  The short last block (Tl
    // 64-k sub-tiles) gives it 4 Tl bytes at 4 Tl l; it is read through a 16-byte window moved back to end inside the
    // block, shifted into place and cleared past K before the transpose (zero codes: the activation bytes past K
    // add nothing).  Row groups past N load a real row group (never stored).
    const int Tl = nkb > nfull ? (K - nfull * kBK) / kSubK : 4;
    // with WN < 4 the records of one (column, parity, lane) are shared by 4 / WN threads, kWPer tiles each
    const int w_combo = tid % (WN * 128), w_ni0 = (tid / (WN * 128)) * kWPer;
    const int w_col = w_combo >> 7, w_par = (w_combo >> 6) & 1, w_l = lane;
    const int w_chunk = 16 * (2 * w_par + (w_l >> 5)) + (w_l & 15);          // layout lane chunk l
    const int w_want = 4 * Tl * w_chunk;
    const int w_off_tail = min(w_want, 256 * Tl - 16);
    const int w_sh = (w_want - w_off_tail) >> 2;
    v4u w_reg[kWPer];
    uint32_t w_rgb[kWPer];
#pragma unroll
    for (int i = 0; i < kWPer; ++i) {
        const int rgl = 8 * w_col + 2 * (w_ni0 + i) + ((w_l >> 4) & 1);
        w_rgb[i] = (uint32_t)min(rg0 + rgl, nrg - 1) * (4u * (uint32_t)K);
    }
    auto load_w = [&](int kb) {
        const uint8_t* pk = packed + (size_t)kb * 1024;
        const uint32_t off = kb < nfull ? 16u * (uint32_t)w_chunk : (uint32_t)w_off_tail;
#pragma unroll
        for (int i = 0; i < kWPer; ++i) w_reg[i] = *reinterpret_cast<const v4u*>(pk + (w_rgb[i] + off));
    };
    // Record j (step 2 j + parity) of this thread.  The window shift is a two-step barrel shift on the bits of the
    // lane's word shift, all selects: a branch (or a compare chain, which the compiler turns into one) here makes it
    // wait for every load in flight where the paths join.
    auto store_w1 = [&](int buf, bool full, int j) {
        const int sh = full ? 0 : w_sh;
        const bool s1 = (sh & 1) != 0, s2 = (sh & 2) != 0;
        const bool live = full || j < Tl;
        uint32_t rec[kWPer];
#pragma unroll
        for (int i = 0; i < kWPer; ++i) {
            const v4u w = w_reg[i];
            const uint32_t u0 = s1 ? w.y : w.x, u1 = s1 ? w.z : w.y, u2 = s1 ? w.w : w.z, u3 = w.w;
            const uint32_t t0 = s2 ? u2 : u0, t1 = s2 ? u3 : u1;
            const uint32_t wj = j == 0 ? t0 : j == 1 ? t1 : j == 2 ? u2 : u3;
            rec[i] = live ? wj : 0u;
        }
        uint32_t* dst = reinterpret_cast<uint32_t*>(&Ws[buf][(w_col * 8 + 2 * j + w_par) * 64 + w_l]) + w_ni0;
        if constexpr (kWPer == 4) *reinterpret_cast<v4u*>(dst) = v4u{rec[0], rec[1], rec[2], rec[3]};
        else *reinterpret_cast<uint2*>(dst) = make_uint2(rec[0], rec[1]);
    };
    auto store_w = [&](int buf, bool full) {
#pragma unroll
        for (int j = 0; j < 4; ++j) store_w1(buf, full, j);
    };

    // ---- the MFMAs of one stage: 8 steps of 32 k ----
    v16i acc[MT][NT];
#pragma unroll
    for (int mi = 0; mi < MT; ++mi)
#pragma unroll
        for (int ni = 0; ni < NT; ++ni) acc[mi][ni] = v16i{};
    int rs_part[MT] = {0, 0};
    // activation operand of step s, tile mi: token row 64 wm + 32 mi + j, bytes 32 s + 16 h of the stage
    const int a_lane = (64 * wm + j32) * kARow + 16 * h;
    const int w_lane = wn * 8 * 64 + lane;
    // (steps at or past `live` lie past K: their activation bytes are not real codes and stay out of the sums)
    // The activation operands of step s + 1 are read while step s multiplies (two register sets), so a wave never
    // waits on LDS between steps; the sched barriers keep the compiler from moving the reads back to their use.
    auto mac_stage = [&](int buf, int live, auto&& after_step) {
        const int s0 = wk * kSteps;                               // this K-group's first k-step of the stage
        v4i a[2][MT];
        v4u b[2];
#pragma unroll
        for (int mi = 0; mi < MT; ++mi)
            a[0][mi] = *reinterpret_cast<const v4i*>(As[buf] + a_lane + 32 * kARow * mi + 32 * s0);
        b[0] = Ws[buf][w_lane + 64 * s0];
#pragma unroll
        for (int i = 0; i < kSteps; ++i) {
            const int cur = i & 1, s = s0 + i;
            if (i + 1 < kSteps) {
#pragma unroll
                for (int mi = 0; mi < MT; ++mi)
                    a[cur ^ 1][mi] = *reinterpret_cast<const v4i*>(As[buf] + a_lane + 32 * kARow * mi + 32 * (s + 1));
                b[cur ^ 1] = Ws[buf][w_lane + 64 * (s + 1)];
            }
            __builtin_amdgcn_sched_barrier(0);
            if (!HAS_RS && wn == 0) {
#pragma unroll
                for (int mi = 0; mi < MT; ++mi)
                    rs_part[mi] = s < live ? byte_sum(a[cur][mi], rs_part[mi]) : rs_part[mi];
            }
#pragma unroll
            for (int ni = 0; ni < NT; ++ni) {
                const v4i bq = unpack_codes(word_of(b[cur], ni));
#pragma unroll
                for (int mi = 0; mi < MT; ++mi)
                    acc[mi][ni] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[cur][mi], bq, acc[mi][ni], 0, 0, 0);
            }
            after_step(i);
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // Stage kb is in LDS buffer (kb - kb_lo) % 2.  Each stage starts with a barrier (its operands are in LDS and
    // everyone finished the previous stage); while its MFMAs run, each thread writes the next stage's chunks (loaded
    // a whole stage earlier) into the other buffer, one after each 32-k step, and reloads each register with the
    // stage after: the waves sharing a SIMD then always have MFMAs to issue while the copies drain.  Stage indices
    // past the slice are clamped to its last stage: those loads repeat it and nothing is computed from them.
    static_assert(kAChunks == 4, "four activation chunks per thread per stage");
    // copies per step: WK = 1 spreads the 4 activation chunks over steps 0-3 and the 4 weight records over 4-7;
    // WK = 2 does one of each per step
    constexpr int kWStep = kSteps == 8 ? 4 : 0;
    const int last = kb_hi - 1;
    if (kb_lo < kb_hi) {
        load_a(kb_lo);
        load_w(kb_lo);
        store_a(0);
        store_w(0, kb_lo < nfull);
        load_a(min(kb_lo + 1, last));
        load_w(min(kb_lo + 1, last));
        int buf = 0;
        for (int kb = kb_lo; kb < kb_hi; ++kb) {
            __syncthreads();
            const int nxt = min(kb + 1, last), nxt2 = min(kb + 2, last);
            const bool nxt_full = nxt < nfull;
            mac_stage(buf, kb < nfull ? 8 : 2 * Tl, [&](int i) {
                if (i < kAChunks) {
                    store_a1(buf ^ 1, i);
                    load_a1(nxt2, i);
                }
                if (i >= kWStep) store_w1(buf ^ 1, nxt_full, i - kWStep);
                if (i == kSteps - 1) load_w(nxt2);
            });
            buf ^= 1;
        }
    }

    // The K-groups past the first hand their partial tiles to the first through LDS (the staging buffers are free
    // once every wave has passed the barrier below).  Token sums: from x_rowsum, or each K-group's partial from its
    // activation operands.  Every wave passes every barrier up to the split-K return.
    __syncthreads();
    v4i* red = reinterpret_cast<v4i*>(smem);                      // [wave tile][mi][ni][4 words][lane]
    const int slot = (wm * WN + wn) * (MT * NT * 4);
    if (WK > 1 && wk == 1) {
#pragma unroll
        for (int mi = 0; mi < MT; ++mi)
#pragma unroll
            for (int ni = 0; ni < NT; ++ni)
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4)
                    red[(slot + (mi * NT + ni) * 4 + q4) * 64 + lane] =
                        v4i{acc[mi][ni][4 * q4], acc[mi][ni][4 * q4 + 1], acc[mi][ni][4 * q4 + 2], acc[mi][ni][4 * q4 + 3]};
    }
    if (HAS_RS) {
        if (tid < kBM) rowsum_s[0][tid] = (m0 + tid < M) ? x_rowsum[m0 + tid] : 0;
    } else if (wn == 0) {
        // lanes j and j + 32 summed the two halves of token row 64 wm + 32 mi + j over this K-group's steps
#pragma unroll
        for (int mi = 0; mi < MT; ++mi) {
            const int v = rs_part[mi] + __shfl_xor(rs_part[mi], 32, 64);
            if (h == 0) rowsum_s[wk][64 * wm + 32 * mi + j32] = v;
        }
    }
    __syncthreads();
    if (WK > 1 && wk == 0) {
#pragma unroll
        for (int mi = 0; mi < MT; ++mi)
#pragma unroll
            for (int ni = 0; ni < NT; ++ni)
#pragma unroll
                for (int q4 = 0; q4 < 4; ++q4) {
                    const v4i o = red[(slot + (mi * NT + ni) * 4 + q4) * 64 + lane];
                    acc[mi][ni][4 * q4] += o.x;
                    acc[mi][ni][4 * q4 + 1] += o.y;
                    acc[mi][ni][4 * q4 + 2] += o.z;
                    acc[mi][ni][4 * q4 + 3] += o.w;
                }
    }

    if (part) {
        // split-K: this slice's exact partial sums (the code offset and the scales are applied when the slices
        // are summed)
        if (wk != 0) return;
        int32_t* pp = part + (size_t)split * M * P.n_total;
#pragma unroll
        for (int mi = 0; mi < MT; ++mi)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int m = m0 + 64 * wm + 32 * mi + 8 * (v >> 2) + 4 * h + (v & 3);
                if (m >= M) continue;
#pragma unroll
                for (int ni = 0; ni < NT; ++ni) {
                    const int n = n0 + 128 * wn + 32 * ni + j32;
                    if (n < N) pp[(size_t)m * N + n] = acc[mi][ni][v];
                }
            }
        return;
    }

    // Epilogue in two passes of 64 token rows (MFMA row tile mi of both wave rows): the waves holding the sums
    // write y = (acc - sum_k xq) * beta / s_m into LDS (row stride kBN + 8 floats: the two half-waves of a write
    // land on different banks), then every thread copies whole 16-byte runs of rows out, so a wave's store is
    // 1 KiB of one output row.  The stores carry the streaming hint: nothing here reads y again.
    // D element v of lane (j, h): row 8 (v / 4) + 4 h + v % 4, column j (weight row n0 + 128 wn + 32 ni + j).
    typedef float v4f __attribute__((ext_vector_type(4)));
    constexpr int kYRow = kBN + 8;
    static_assert(64 * kYRow * 4 <= kSmem, "one pass of the output tile fits the staging LDS");
    float* ybuf = reinterpret_cast<float*>(smem);
    const float beta = *w_scale;
    constexpr int kQuads = 64 * kBN / 4, kQPerRow = kBN / 4;
#pragma unroll
    for (int mi = 0; mi < MT; ++mi) {
        __syncthreads();                                          // LDS free: partial tiles or the previous pass read
        if (wk == 0) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int rr = 8 * (v >> 2) + 4 * h + (v & 3);
                const int ml = 64 * wm + 32 * mi + rr;
                const int m = min(m0 + ml, M - 1);
                int rsum = rowsum_s[0][ml];
                if (!HAS_RS) {
#pragma unroll
                    for (int g = 1; g < WK; ++g) rsum += rowsum_s[g][ml];
                }
                const float sc = beta / x_scale[m];
#pragma unroll
                for (int ni = 0; ni < NT; ++ni) {
                    const int nl = 128 * wn + 32 * ni + j32;
                    const int val = acc[mi][ni][v] - rsum;
                    ybuf[(32 * wm + rr) * kYRow + nl] = (float)val * sc;
                    if constexpr (HAS_ACC) {
                        if (acc_out && m0 + ml < M && n0 + nl < N) acc_out[(size_t)(m0 + ml) * N + n0 + nl] = val;
                    }
                }
            }
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < kQuads / kThreads; ++i) {
            const int f = tid + i * kThreads;
            const int lr = f / kQPerRow, c4 = f - lr * kQPerRow;
            const int m = m0 + 64 * (lr >> 5) + 32 * mi + (lr & 31);
            const int n = n0 + 4 * c4;
            if (m < M && n < N) {
                const v4f o = *reinterpret_cast<const v4f*>(ybuf + lr * kYRow + 4 * c4);
                __builtin_nontemporal_store(o, reinterpret_cast<v4f*>(y + (size_t)m * N + n));
            }
        }
    }
}

// Sum of the split-K slices, then the epilogue y = (sum - sum_k xq[m, k]) * (beta / s_m), for every weight of the
// launch in one pass: output quad i4 belongs to the weight whose run of M N / 4 quads holds it (a scalar-free
// compare chain over the fixed maximum).  Each weight's block in a slice starts at its part offset; slices are
// `slice` words apart.
struct FinishLinears {
    float* y[kMaxFused];
    int32_t* acc[kMaxFused];
    const float* w_scale[kMaxFused];
    long long part_off[kMaxFused];
    long long start4[kMaxFused];      // first output quad of each weight; LLONG_MAX past the last
    int N[kMaxFused];
    long long total4;
};

__global__ __launch_bounds__(256) void prefill_splitk_finish(FinishLinears F, const int32_t* __restrict__ part,
                                                             int64_t slice, int splits,
                                                             const int32_t* __restrict__ x_rowsum,
                                                             const float* __restrict__ x_scale) {
    const int64_t i4 = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i4 >= F.total4) return;
    int li = 0;
#pragma unroll
    for (int i = 1; i < kMaxFused; ++i) li = i4 >= F.start4[i] ? i : li;
    const int64_t local = i4 - pick_linear(F.start4, li);
    const int N = pick_linear(F.N, li);
    const int m = (int)(local / (N >> 2));
    const size_t off = (size_t)pick_linear(F.part_off, li) + (size_t)local * 4;
    v4i t = *reinterpret_cast<const v4i*>(part + off);
    for (int sp = 1; sp < splits; ++sp) t += *reinterpret_cast<const v4i*>(part + (size_t)sp * slice + off);
    const int rs = x_rowsum[m];
    t -= (v4i){rs, rs, rs, rs};
    const float sc = *pick_linear(F.w_scale, li) / x_scale[m];
    typedef float v4f __attribute__((ext_vector_type(4)));
    const v4f o = {(float)t.x * sc, (float)t.y * sc, (float)t.z * sc, (float)t.w * sc};
    __builtin_nontemporal_store(o, reinterpret_cast<v4f*>(pick_linear(F.y, li) + (size_t)local * 4));
    int32_t* acc_out = pick_linear(F.acc, li);
    if (acc_out) *reinterpret_cast<v4i*>(acc_out + (size_t)local * 4) = t;
}

// Tile width and split-K factor for the weight tiles of a launch.  Whichever of the 128 x 512 and 128 x 256 tiles
// (two K-groups) needs fewer rounds of work groups over the CUs, weighting a round of the narrow tile at 0.84 of a
// wide one (measured at K = 4096 and 14336).  Splitting K keeps still smaller grids busy: as many slices as keep
// one round (at least two 256-k stages per slice), only for grids that leave at least half the CUs idle (the
// slices' extra pass over M x N costs more elsewhere).
void prefill_plan(const FusedLinears& L, int64_t M, int64_t K, int& wn, int& splits) {
    const int64_t cus = device_cus();
    const int64_t tiles_m = (M + kBM - 1) / kBM;
    int64_t n4 = 0, n2 = 0;
    for (int i = 0; i < L.count; ++i) {
        n4 += (L.N[i] + 511) / 512;
        n2 += (L.N[i] + 255) / 256;
    }
    const int64_t r4 = (tiles_m * n4 + cus - 1) / cus, r2 = (tiles_m * n2 + cus - 1) / cus;
    wn = r2 * 84 < r4 * 100 ? 2 : 4;
    const int64_t tiles = tiles_m * (wn == 4 ? n4 : n2);
    const int64_t nkb = (K + kBK - 1) / kBK;
    int64_t sp = 2 * tiles <= cus ? cus / tiles : 1;
    if (sp > nkb / 2) sp = nkb / 2;
    if (sp > kMaxSplits) sp = kMaxSplits;
    splits = sp > 1 ? (int)sp : 1;
    // slices of whole stages: no empty slice
    if (splits > 1) {
        const int64_t per = (nkb + splits - 1) / splits;
        splits = (int)((nkb + per - 1) / per);
    }
}

int64_t total_rows(const FusedLinears& L) {
    int64_t n = 0;
    for (int i = 0; i < L.count; ++i) n += L.N[i];
    return n;
}

template <int WN>
void launch_wn(const FusedLinears& L, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum, int M, int K,
               int splits, int32_t* part, hipStream_t stream) {
    PrefillLinears P{};
    int tiles = 0;
    long long off = 0;
    for (int i = 0; i < kMaxFused; ++i) {
        if (i < L.count) {
            P.packed[i] = L.packed[i];
            P.w_scale[i] = L.w_scale[i];
            P.y[i] = L.y[i];
            P.acc[i] = L.acc[i];
            P.N[i] = L.N[i];
            P.part_off[i] = off;
            P.tile_start[i] = tiles;
            P.tile_start_lo[i] = tiles;
            off += (long long)M * L.N[i];
            tiles += (L.N[i] + 128 * WN - 1) / (128 * WN);
        } else {
            P.packed[i] = L.packed[0];
            P.w_scale[i] = L.w_scale[0];
            P.y[i] = L.y[0];
            P.acc[i] = L.acc[0];
            P.N[i] = L.N[0];
            P.part_off[i] = 0;
            P.tile_start[i] = 0x7fffffff;
            P.tile_start_lo[i] = 0;
        }
    }
    P.tile_start[kMaxFused] = 0x7fffffff;
    P.tiles_n = tiles;
    P.n_total = total_rows(L);
    const unsigned grid_tiles = (unsigned)(((M + kBM - 1) / kBM) * tiles);
    const dim3 grid(grid_tiles * (unsigned)splits), block(kThreads);
    bool has_acc = false;
    for (int i = 0; i < L.count; ++i) has_acc = has_acc || L.acc[i] != nullptr;
    if (x_rowsum && has_acc)
        hipLaunchKernelGGL((i2s_prefill_kernel<WN, true, true>), grid, block, 0, stream, P, xq, x_scale, x_rowsum, M,
                           K, splits, part);
    else if (x_rowsum)
        hipLaunchKernelGGL((i2s_prefill_kernel<WN, true, false>), grid, block, 0, stream, P, xq, x_scale, x_rowsum, M,
                           K, splits, part);
    else if (has_acc)
        hipLaunchKernelGGL((i2s_prefill_kernel<WN, false, true>), grid, block, 0, stream, P, xq, x_scale, x_rowsum, M,
                           K, splits, part);
    else
        hipLaunchKernelGGL((i2s_prefill_kernel<WN, false, false>), grid, block, 0, stream, P, xq, x_scale, x_rowsum, M,
                           K, splits, part);
}

}  // namespace

size_t prefill_workspace_bytes(const FusedLinears& L, int64_t M, int64_t K) {
    int wn, splits;
    prefill_plan(L, M, K, wn, splits);
    return splits > 1 ? (size_t)splits * (size_t)M * (size_t)total_rows(L) * sizeof(int32_t) : 0;
}

hipError_t launch_i2s_prefill(const FusedLinears& L, const int8_t* xq, const float* x_scale, const int32_t* x_rowsum,
                              int M, int K, void* ws, size_t ws_bytes, hipStream_t stream) {
    int wn, splits;
    prefill_plan(L, M, K, wn, splits);
    const int64_t ntot = total_rows(L);
    // split-K needs the token sums and the workspace for the slices
    if (!x_rowsum || !ws || ws_bytes < (size_t)splits * M * ntot * sizeof(int32_t)) splits = 1;
    int32_t* part = splits > 1 ? static_cast<int32_t*>(ws) : nullptr;
    if (wn == 4)
        launch_wn<4>(L, xq, x_scale, x_rowsum, M, K, splits, part, stream);
    else
        launch_wn<2>(L, xq, x_scale, x_rowsum, M, K, splits, part, stream);
    if (splits > 1) {
        FinishLinears F{};
        int64_t off = 0, q4 = 0;
        for (int i = 0; i < kMaxFused; ++i) {
            const bool live = i < L.count;
            F.y[i] = L.y[live ? i : 0];
            F.acc[i] = L.acc[live ? i : 0];
            F.w_scale[i] = L.w_scale[live ? i : 0];
            F.N[i] = L.N[live ? i : 0];
            F.part_off[i] = live ? off : 0;
            F.start4[i] = live ? q4 : 0x7fffffffffffffffLL;
            if (live) {
                off += (int64_t)M * L.N[i];
                q4 += (int64_t)M * (L.N[i] / 4);
            }
        }
        F.total4 = q4;
        hipLaunchKernelGGL(prefill_splitk_finish, dim3((unsigned)((q4 + 255) / 256)), dim3(256), 0, stream, F, part,
                           (int64_t)M * ntot, splits, x_rowsum, x_scale);
    }
    return hipGetLastError();
}

}  // namespace bitnet
