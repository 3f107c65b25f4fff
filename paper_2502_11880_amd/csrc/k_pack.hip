// Offline weight preprocessing: absmean ternarisation (Sec. 2.1) and packing into the I2_S format
// (Table 1, Sec. 3.2.2) or the TL2 format (Sec. 3.1: mirror consolidation, signed-unsigned weight
// splitting, block-fitting weight splitting; codes of Table 5 and Table 6).
//
// beta is the fp32 value nearest to the exact mean of |W| (ties to even), so it is the same for any
// launch shape and summation order:
//   1. every |w| = m * 2^(e-150) (24-bit significand m, biased exponent e; subnormals use e = 1);
//      significands are summed exactly into 256 uint64 buckets, one per exponent (LDS, then global);
//   2. one thread folds the buckets into a 384-bit integer T (sum |w| = T * 2^-149), divides T * 2^64
//      by N*K with 32-bit limbs, and rounds the quotient to 24 significant bits, ties to even.
#include "bitnet_internal.hpp"

namespace bitnet {
namespace {

constexpr int kBuckets = 256;

__global__ __launch_bounds__(256) void fill_zero_u64(unsigned long long* p, int n) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0ull;
}

__device__ __forceinline__ void bucket_add(unsigned long long* sb, float w) {
    const uint32_t bits = __float_as_uint(w) & 0x7FFFFFFFu;
    const uint32_t e = bits >> 23;
    const uint32_t f = bits & 0x7FFFFFu;
    const uint32_t m = e ? (f | 0x800000u) : f;
    if (m) atomicAdd(&sb[e ? e : 1u], (unsigned long long)m);
}

__global__ __launch_bounds__(256) void absmean_buckets(const float4* __restrict__ W4, size_t n4,
                                                       unsigned long long* __restrict__ buckets) {
    __shared__ unsigned long long sb[kBuckets];
    sb[threadIdx.x] = 0ull;
    __syncthreads();
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (size_t)gridDim.x * 256) {
        const float4 v = W4[i];
        bucket_add(sb, v.x);
        bucket_add(sb, v.y);
        bucket_add(sb, v.z);
        bucket_add(sb, v.w);
    }
    __syncthreads();
    const unsigned long long s = sb[threadIdx.x];
    if (s) atomicAdd(&buckets[threadIdx.x], s);
}

// ---- multi-limb helpers (little-endian 32-bit limbs) ----
__device__ void limbs_add_shifted(uint32_t* T, int nlimbs, unsigned long long v, int sh) {
    const int li = sh >> 5, bi = sh & 31;
    const uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
    uint32_t parts[3];
    if (bi == 0) {
        parts[0] = lo; parts[1] = hi; parts[2] = 0u;
    } else {
        parts[0] = lo << bi;
        parts[1] = (lo >> (32 - bi)) | (hi << bi);
        parts[2] = hi >> (32 - bi);
    }
    unsigned long long carry = 0;
    for (int i = li; i < nlimbs; ++i) {
        const int d = i - li;
        if (d >= 3 && carry == 0) break;
        const unsigned long long add = d < 3 ? parts[d] : 0u;
        const unsigned long long s = (unsigned long long)T[i] + add + carry;
        T[i] = (uint32_t)s;
        carry = s >> 32;
    }
}

__device__ __forceinline__ uint32_t limbs_bit(const uint32_t* Q, int pos) {
    return (Q[pos >> 5] >> (pos & 31)) & 1u;
}

__global__ void absmean_finalize(const unsigned long long* __restrict__ buckets, unsigned long long count,
                                 float* __restrict__ beta_out) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    constexpr int kT = 12;          // 384 bits: bucket b adds at most 2^55 * 2^(b-1) < 2^309
    constexpr int kU = kT + 2;      // T * 2^64
    uint32_t U[kU];
    for (int i = 0; i < kU; ++i) U[i] = 0u;
    bool any = false;
    for (int b = 1; b < kBuckets; ++b) {
        const unsigned long long s = buckets[b];
        if (!s) continue;
        any = true;
        limbs_add_shifted(U, kU, s, (b - 1) + 64);
    }
    if (!any) {
        *beta_out = 0.0f;
        return;
    }
    // Q = floor(U / count), remainder -> sticky.  count < 2^32, so each step divides a 64-bit value.
    uint32_t Q[kU];
    unsigned long long rem = 0;
    for (int i = kU - 1; i >= 0; --i) {
        const unsigned long long cur = (rem << 32) | U[i];
        Q[i] = (uint32_t)(cur / count);
        rem = cur % count;
    }
    const bool sticky_rem = rem != 0;
    int top = kU - 1;
    while (top > 0 && Q[top] == 0u) --top;
    const int p = top * 32 + 31 - __clz((int)Q[top]);   // highest set bit; value = Q * 2^-213
    const int E = p - 213;
    const int shift = (E >= -126) ? p - 23 : 64;
    uint32_t mant = 0;
    for (int i = 23; i >= 0; --i) {
        const int pos = shift + i;
        mant = (mant << 1) | (pos < kU * 32 ? limbs_bit(Q, pos) : 0u);
    }
    const uint32_t half = limbs_bit(Q, shift - 1);
    bool lower = sticky_rem;
    for (int pos = 0; pos < shift - 1 && !lower; ++pos) lower = limbs_bit(Q, pos) != 0u;
    if (half && (lower || (mant & 1u))) mant += 1u;
    uint32_t bits;
    if (E >= -126) bits = ((uint32_t)(E + 126) << 23) + mant;   // mant in [2^23, 2^24]
    else bits = mant;                                             // subnormal (mant <= 2^23)
    *beta_out = __uint_as_float(bits);
}

__device__ __forceinline__ int ternary(float w, float beta) {
    if (beta == 0.0f) return 0;
    const float r = rintf(w / beta);       // IEEE divide, ties-to-even rounding
    return (int)fminf(fmaxf(r, -1.0f), 1.0f);
}

// I2_S: one thread per packed 32-bit word (16 weights of one row).
__global__ __launch_bounds__(256) void pack_i2s_words(const float* __restrict__ W, int K, size_t nwords,
                                                      const float* __restrict__ beta_p,
                                                      uint32_t* __restrict__ out) {
    const size_t d = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (d >= nwords) return;
    const float beta = *beta_p;
    const size_t R = d / (size_t)K;                   // a row group holds K words (4K bytes)
    const int rem = (int)(d - R * (size_t)K);
    const int s = rem >> 8;                           // 1 KiB blocks of 256 words
    const int w = rem & 255;
    const int nsub = K / kSubK;
    const int T = min(4, nsub - 4 * s);
    const int l = w / T, j = w - l * T;
    const int r = l & 15, q = l >> 4;
    const size_t n = R * kRowsPerGroup + r;
    const int k0 = kSubK * (4 * s + j) + 16 * q;
    const float4* src = reinterpret_cast<const float4*>(W + n * (size_t)K + k0);
    uint32_t word = 0;
#pragma unroll
    for (int f = 0; f < 4; ++f) {
        const float4 v = src[f];                      // k0 + 4f + b, b = 0..3
        word |= (uint32_t)(ternary(v.x, beta) + 1) << (2 * f);
        word |= (uint32_t)(ternary(v.y, beta) + 1) << (8 + 2 * f);
        word |= (uint32_t)(ternary(v.z, beta) + 1) << (16 + 2 * f);
        word |= (uint32_t)(ternary(v.w, beta) + 1) << (24 + 2 * f);
    }
    out[d] = word;
}

// TL1 (Algorithm TL1, Table 5): the I2_S tiling, one thread per 32-bit word = 8 pair codes (16 weights) of one row;
// pair i (weights k0 + 2i, k0 + 2i + 1) in byte i % 4, low nibble for i < 4, high nibble for i >= 4.
__global__ __launch_bounds__(256) void pack_tl1_words(const float* __restrict__ W, int K, size_t nwords,
                                                      const float* __restrict__ beta_p,
                                                      uint32_t* __restrict__ out) {
    const size_t d = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (d >= nwords) return;
    const float beta = *beta_p;
    const size_t R = d / (size_t)K;                   // a row group holds K words (4K bytes)
    const int rem = (int)(d - R * (size_t)K);
    const int s = rem >> 8;                           // 1 KiB blocks of 256 words
    const int w = rem & 255;
    const int nsub = K / kSubK;
    const int T = min(4, nsub - 4 * s);
    const int l = w / T, j = w - l * T;
    const int r = l & 15, q = l >> 4;
    const size_t n = R * kRowsPerGroup + r;
    const int k0 = kSubK * (4 * s + j) + 16 * q;
    const float2* src = reinterpret_cast<const float2*>(W + n * (size_t)K + k0);
    uint32_t word = 0;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float2 v = src[i];
        const uint32_t c = (uint32_t)(3 * (ternary(v.x, beta) + 1) + (ternary(v.y, beta) + 1));
        word |= c << (8 * (i & 3) + 4 * (i >> 2));
    }
    out[d] = word;
}

// TL1 words rewritten as I2_S words at the same positions (both formats tile a word as 16 weights of one row):
// weight e of the word is pair e / 2, code c: t + 1 = c / 3 for even e, c % 3 for odd e; it goes to byte e % 4,
// bits 2 (e / 4).  blockIdx.y is the weight.
struct Tl1Transcode {
    const uint32_t* src[kMaxFused];
    uint32_t* dst[kMaxFused];
    size_t nwords[kMaxFused];
};

__global__ __launch_bounds__(256) void tl1_to_i2s_words(Tl1Transcode T) {
    const int li = blockIdx.y;
    const size_t d = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (d >= T.nwords[li]) return;
    const uint32_t w = T.src[li][d];
    uint32_t o = 0;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
        const int i = e >> 1;
        const uint32_t c = (w >> (8 * (i & 3) + 4 * (i >> 2))) & 0xFu;
        const uint32_t code = (e & 1) ? c % 3u : c / 3u;
        o |= code << (8 * (e & 3) + 2 * (e >> 2));
    }
    T.dst[li][d] = o;
}

// TL2 part: one thread per lane chunk = 32 triples (96 weights) of one row in one 384-k block.
__global__ __launch_bounds__(256) void pack_tl2_chunks(const float* __restrict__ W, int K, int nblk,
                                                       size_t nchunks, const float* __restrict__ beta_p,
                                                       uint32_t* __restrict__ idx_plane,
                                                       uint32_t* __restrict__ sign_plane) {
    const size_t c = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (c >= nchunks) return;
    const float beta = *beta_p;
    const size_t rb = c >> 6;                         // (row group, block) pair
    const int l = (int)(c & 63);
    const size_t R = rb / (size_t)nblk;
    const int blk = (int)(rb - R * (size_t)nblk);
    const int r = l & 15, q = l >> 4;
    const size_t n = R * kRowsPerGroup + r;
    const float* src = W + n * (size_t)K + (size_t)blk * kTl2BlockK + 96 * q;
    uint32_t idxw[4] = {0u, 0u, 0u, 0u};
    uint32_t sign = 0u;
    for (int i = 0; i < 32; ++i) {
        const int t0 = ternary(src[3 * i], beta), t1 = ternary(src[3 * i + 1], beta),
                  t2 = ternary(src[3 * i + 2], beta);
        const int v = 9 * t0 + 3 * t1 + t2;
        const uint32_t a = (uint32_t)(v < 0 ? -v : v);
        idxw[i >> 3] |= a << (4 * (i & 7));
        sign |= (uint32_t)(v < 0) << i;
    }
    uint4 o;
    o.x = idxw[0]; o.y = idxw[1]; o.z = idxw[2]; o.w = idxw[3];
    reinterpret_cast<uint4*>(idx_plane)[c] = o;
    sign_plane[c] = sign;
}

// TL1 tail: one thread per 32-bit word = 8 pairs (16 weights) of one row.
__global__ __launch_bounds__(256) void pack_tl1_tail(const float* __restrict__ W, int K, int three, int units,
                                                     size_t nwords, const float* __restrict__ beta_p,
                                                     uint32_t* __restrict__ tail) {
    const size_t d = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (d >= nwords) return;
    const float beta = *beta_p;
    const size_t per_rg = (size_t)64 * units;
    const size_t R = d / per_rg;
    const int rem = (int)(d - R * per_rg);
    const int l = rem / units, u = rem - l * units;
    const int r = l & 15, q = l >> 4;
    const size_t n = R * kRowsPerGroup + r;
    const float* src = W + n * (size_t)K + three + kSubK * u + 16 * q;
    uint32_t word = 0;
    for (int i = 0; i < 8; ++i) {
        const int t0 = ternary(src[2 * i], beta), t1 = ternary(src[2 * i + 1], beta);
        word |= (uint32_t)(3 * (t0 + 1) + (t1 + 1)) << (4 * i);
    }
    tail[d] = word;
}

inline unsigned grid_for(size_t n, int block) { return (unsigned)((n + block - 1) / block); }

}  // namespace

size_t pack_workspace_bytes() { return kBuckets * sizeof(unsigned long long); }

hipError_t launch_pack(int layout, const float* W, int64_t N, int64_t K, void* packed, float* w_scale,
                       void* ws, hipStream_t stream) {
    unsigned long long* buckets = static_cast<unsigned long long*>(ws);
    hipLaunchKernelGGL(fill_zero_u64, dim3(1), dim3(256), 0, stream, buckets, kBuckets);
    const size_t n = (size_t)N * (size_t)K;
    const size_t n4 = n / 4;
    const unsigned gb = (unsigned)std::min<size_t>(2048, (n4 + 255) / 256);
    hipLaunchKernelGGL(absmean_buckets, dim3(gb), dim3(256), 0, stream,
                       reinterpret_cast<const float4*>(W), n4, buckets);
    hipLaunchKernelGGL(absmean_finalize, dim3(1), dim3(64), 0, stream, buckets, (unsigned long long)n,
                       w_scale);
    if (layout == 0) {
        const size_t nwords = n / 16;
        hipLaunchKernelGGL(pack_i2s_words, dim3(grid_for(nwords, 256)), dim3(256), 0, stream, W, (int)K,
                           nwords, w_scale, static_cast<uint32_t*>(packed));
    } else if (layout == 2) {
        const size_t nwords = n / 16;
        hipLaunchKernelGGL(pack_tl1_words, dim3(grid_for(nwords, 256)), dim3(256), 0, stream, W, (int)K,
                           nwords, w_scale, static_cast<uint32_t*>(packed));
    } else {
        const int three = (int)(K / kTl2BlockK) * kTl2BlockK;
        const int two = (int)K - three;
        uint8_t* base = static_cast<uint8_t*>(packed);
        uint32_t* idx_plane = reinterpret_cast<uint32_t*>(base);
        uint32_t* sign_plane = reinterpret_cast<uint32_t*>(base + (size_t)N * three / 6);
        uint32_t* tail = reinterpret_cast<uint32_t*>(base + (size_t)N * three / 6 + (size_t)N * three / 24);
        if (three) {
            const int nblk = three / kTl2BlockK;
            const size_t nchunks = (size_t)(N / kRowsPerGroup) * nblk * 64;
            hipLaunchKernelGGL(pack_tl2_chunks, dim3(grid_for(nchunks, 256)), dim3(256), 0, stream, W,
                               (int)K, nblk, nchunks, w_scale, idx_plane, sign_plane);
        }
        if (two) {
            const int units = two / kSubK;
            const size_t nwords = (size_t)(N / kRowsPerGroup) * 64 * units;
            hipLaunchKernelGGL(pack_tl1_tail, dim3(grid_for(nwords, 256)), dim3(256), 0, stream, W, (int)K,
                               three, units, nwords, w_scale, tail);
        }
    }
    return hipGetLastError();
}

hipError_t launch_tl1_to_i2s(const void* const* packed, const int* N, void* const* i2s_out, int count, int K,
                             hipStream_t stream) {
    Tl1Transcode T{};
    size_t most = 0;
    for (int i = 0; i < count; ++i) {
        T.src[i] = static_cast<const uint32_t*>(packed[i]);
        T.dst[i] = static_cast<uint32_t*>(i2s_out[i]);
        T.nwords[i] = (size_t)N[i] * (size_t)K / 16;
        most = T.nwords[i] > most ? T.nwords[i] : most;
    }
    hipLaunchKernelGGL(tl1_to_i2s_words, dim3(grid_for(most, 256), (unsigned)count), dim3(256), 0, stream, T);
    return hipGetLastError();
}

}  // namespace bitnet
