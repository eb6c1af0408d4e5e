// Windowed single-token decode for gfx950: split-KV with partial online-softmax
// states and a merge kernel (the decode form of Fig. fa is the last query row;
// the split/merge decomposition is the one Sec. 5 describes), over a
// pair-chunk-major K cache so that pruned pairs are never read from HBM.
//
// K cache layout [B][h_kv][d/16][n_k][16]: chunk c of a head is a contiguous
// stream over tokens of 16 bf16 = dims [8c, 8c+8) then [d/2 + 8c, d/2 + 8c + 8).
// With the query at position q_pos, token t sits at distance z = q_pos - t, and
// chunk c is needed only for z <= max_{r in c} W_r: a contiguous suffix of the
// stream.  Tokens with chunk_min < z <= chunk_max keep some pairs of the chunk;
// the dropped pairs are zeroed per token before the dot product.
//
// Workgroup = 4 waves over one token split of one (batch, kv head, group of
// query heads).  QK: lane = token (64 tokens per wave step), dot products in
// fp32 against the pre-scaled query held in LDS.  PV: lanes re-map to
// (token group, 8 output dims) so V rows stream as 16-byte loads; the per-token
// probabilities pass through LDS.  The split writes (max, normaliser, output)
// partials; decode_merge_kernel combines them.
#include "atf_internal.hpp"

namespace atf {
namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf_lo(uint32_t x) { return __builtin_bit_cast(float, x << 16); }
__device__ __forceinline__ float bf_hi(uint32_t x) { return __builtin_bit_cast(float, x & 0xFFFF0000u); }
__device__ __forceinline__ float bf_to_f(uint16_t x) { return __builtin_bit_cast(float, uint32_t(x) << 16); }
__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
    return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
    return x;
}

constexpr int kWaves = 4;

template <int D, int NG>
__global__ __launch_bounds__(256) void decode_split_kernel(const DecodeParams p) {
    constexpr int kChunks = D / 16;
    constexpr int kHalf = D / 2;
    constexpr int LPT = D / 8;      // lanes per token in the PV phase (8 dims each)
    constexpr int TPI = 64 / LPT;   // tokens per PV load row
    constexpr int ROWS = 64 / TPI;  // PV load rows per 64 tokens

    __shared__ float qs[NG][D];
    __shared__ float ps[kWaves][NG][64];
    __shared__ float red_m[kWaves][NG];
    __shared__ float red_l[kWaves][NG];
    __shared__ float red_o[kWaves][NG][D];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int split = blockIdx.x;
    const int subgroups = p.group / NG;
    const int g = blockIdx.y / subgroups;
    const int sub = blockIdx.y % subgroups;
    const int b = blockIdx.z;
    const int hq0 = g * p.group + sub * NG;

    for (int i = tid; i < NG * D; i += 256) {
        const int h = i / D, x = i % D;
        qs[h][x] = bf_to_f(p.q[(int64_t(b) * p.h_q + hq0 + h) * D + x]) * p.scale_log2;
    }
    __syncthreads();

    const int t_begin = split * p.split_tokens;
    const int t_end = min(p.n_valid, t_begin + p.split_tokens);

    const uint16_t* kstream = p.kpcm + (int64_t(b) * p.h_kv + g) * kChunks * int64_t(p.n_k) * 16;
    const uint16_t* vbase = p.v + (int64_t(b) * p.h_kv + g) * int64_t(p.n_k) * D;

    float m[NG], lpart[NG], o[NG][8];
#pragma unroll
    for (int h = 0; h < NG; ++h) {
        m[h] = -INFINITY;
        lpart[h] = 0.f;
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] = 0.f;
    }

    const int tg = lane / LPT;  // PV token group
    const int ds = lane % LPT;  // PV dims 8*ds .. 8*ds+7

    for (int tb = t_begin + 64 * wave; tb < t_end; tb += 64 * kWaves) {
        // ---- QK: lane = token
        const int t = tb + lane;
        const bool valid = t < t_end;
        const int z = p.q_pos - t;
        const int zmin_wave = p.q_pos - min(tb + 63, t_end - 1);
        float s[NG];
#pragma unroll
        for (int h = 0; h < NG; ++h) s[h] = 0.f;
#pragma unroll
        for (int c = 0; c < kChunks; ++c) {
            const int cmax = p.win.chunk_max[c];
            if (cmax < zmin_wave) continue;  // no token of this wave step keeps the chunk
            if (valid && z <= cmax) {
                const uint16_t* rec = kstream + (int64_t(c) * p.n_k + t) * 16;
                u32x4_t klo = *reinterpret_cast<const u32x4_t*>(rec);
                u32x4_t khi = *reinterpret_cast<const u32x4_t*>(rec + 8);
                if (z > p.win.chunk_min[c]) {  // boundary token: drop pairs with W_r < z
#pragma unroll
                    for (int tt = 0; tt < 4; ++tt) {
                        const uint32_t mk = (z <= p.win.W[8 * c + 2 * tt] ? 0x0000FFFFu : 0u) |
                                            (z <= p.win.W[8 * c + 2 * tt + 1] ? 0xFFFF0000u : 0u);
                        klo[tt] &= mk;
                        khi[tt] &= mk;
                    }
                }
                float kl[8], kh[8];
#pragma unroll
                for (int tt = 0; tt < 4; ++tt) {
                    kl[2 * tt] = bf_lo(klo[tt]);
                    kl[2 * tt + 1] = bf_hi(klo[tt]);
                    kh[2 * tt] = bf_lo(khi[tt]);
                    kh[2 * tt + 1] = bf_hi(khi[tt]);
                }
#pragma unroll
                for (int h = 0; h < NG; ++h) {
                    float acc = s[h];
#pragma unroll
                    for (int e = 0; e < 8; ++e) {
                        acc = __builtin_fmaf(qs[h][8 * c + e], kl[e], acc);
                        acc = __builtin_fmaf(qs[h][kHalf + 8 * c + e], kh[e], acc);
                    }
                    s[h] = acc;
                }
            }
        }
        // ---- online softmax over this wave step (scores already in the log2 domain)
#pragma unroll
        for (int h = 0; h < NG; ++h) {
            const float sv = valid ? s[h] : -INFINITY;
            const float m_new = fmaxf(m[h], wave_max(sv));  // finite: lane 0 is valid
            const float alpha = exp2_fast(m[h] - m_new);
            const float pr = exp2_fast(sv - m_new);
            lpart[h] = lpart[h] * alpha + pr;
#pragma unroll
            for (int e = 0; e < 8; ++e) o[h][e] *= alpha;
            m[h] = m_new;
            ps[wave][h][lane] = pr;
        }
        __builtin_amdgcn_wave_barrier();
        // ---- PV: lanes = (token group, 8 dims)
#pragma unroll 4
        for (int r = 0; r < ROWS; ++r) {
            const int tl = tg * ROWS + r;
            const int tv = tb + tl;
            if (tv < t_end) {
                const u32x4_t vv =
                    *reinterpret_cast<const u32x4_t*>(vbase + int64_t(tv) * D + 8 * ds);
                float vf[8];
#pragma unroll
                for (int tt = 0; tt < 4; ++tt) {
                    vf[2 * tt] = bf_lo(vv[tt]);
                    vf[2 * tt + 1] = bf_hi(vv[tt]);
                }
#pragma unroll
                for (int h = 0; h < NG; ++h) {
                    const float pr = ps[wave][h][tl];
#pragma unroll
                    for (int e = 0; e < 8; ++e) o[h][e] = __builtin_fmaf(pr, vf[e], o[h][e]);
                }
            }
        }
        __builtin_amdgcn_wave_barrier();
    }

    // ---- reduce within the wave, then across waves
#pragma unroll
    for (int h = 0; h < NG; ++h) {
        const float l = wave_sum(lpart[h]);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            float x = o[h][e];
#pragma unroll
            for (int off = LPT; off < 64; off <<= 1) x += __shfl_xor(x, off);
            o[h][e] = x;
        }
        if (lane == 0) {
            red_m[wave][h] = m[h];
            red_l[wave][h] = l;
        }
        if (lane < LPT) {
#pragma unroll
            for (int e = 0; e < 8; ++e) red_o[wave][h][8 * ds + e] = o[h][e];
        }
    }
    __syncthreads();
    for (int i = tid; i < NG * D; i += 256) {
        const int h = i / D, x = i % D;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) M = fmaxf(M, red_m[w][h]);
        float L = 0.f, O = 0.f;
        if (M != -INFINITY) {
#pragma unroll
            for (int w = 0; w < kWaves; ++w) {
                const float f = exp2_fast(red_m[w][h] - M);  // 0 for an idle wave
                L += red_l[w][h] * f;
                O += red_o[w][h][x] * f;
            }
        }
        const int64_t slot = (int64_t(b) * p.h_q + hq0 + h) * p.splits + split;
        if (x == 0) {
            p.ws_m[slot] = M;
            p.ws_l[slot] = L;
        }
        p.ws_o[slot * D + x] = O;
    }
}

template <int D>
__global__ __launch_bounds__(D) void decode_merge_kernel(const DecodeParams p) {
    const int hq = blockIdx.x;
    const int b = blockIdx.y;
    const int x = threadIdx.x;
    const int64_t base = (int64_t(b) * p.h_q + hq) * p.splits;
    float M = -INFINITY;
    for (int s = 0; s < p.splits; ++s) M = fmaxf(M, p.ws_m[base + s]);
    float L = 0.f, O = 0.f;
    for (int s = 0; s < p.splits; ++s) {
        const float ms = p.ws_m[base + s];
        if (ms == -INFINITY) continue;  // split with no causal key
        const float f = exp2_fast(ms - M);
        L += p.ws_l[base + s] * f;
        O += p.ws_o[(base + s) * D + x] * f;
    }
    p.o[(int64_t(b) * p.h_q + hq) * D + x] = __builtin_bit_cast(uint16_t, (__bf16)(O / L));
    if (x == 0) p.lse[int64_t(b) * p.h_q + hq] = M * 0.69314718055994531f + logf(L);
}

template <int D>
__global__ __launch_bounds__(256) void pack_kcache_kernel(const PackParams p) {
    constexpr int kChunks = D / 16;
    const int64_t total = int64_t(p.batch) * p.n_k * p.h_kv * kChunks;
    for (int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x; idx < total;
         idx += int64_t(gridDim.x) * 256) {
        const int c = int(idx % kChunks);
        int64_t r = idx / kChunks;
        const int g = int(r % p.h_kv);
        r /= p.h_kv;
        const int t = int(r % p.n_k);
        const int b = int(r / p.n_k);
        const uint16_t* src = p.src + ((int64_t(b) * p.n_k + t) * p.h_kv + g) * D;
        const u32x4_t lo = *reinterpret_cast<const u32x4_t*>(src + 8 * c);
        const u32x4_t hi = *reinterpret_cast<const u32x4_t*>(src + D / 2 + 8 * c);
        uint16_t* dst = p.dst + (((int64_t(b) * p.h_kv + g) * kChunks + c) * p.n_k + t) * 16;
        *reinterpret_cast<u32x4_t*>(dst) = lo;
        *reinterpret_cast<u32x4_t*>(dst + 8) = hi;
    }
}

template <int D, int NG>
hipError_t launch_split(const DecodeParams& p, hipStream_t stream) {
    const dim3 grid(unsigned(p.splits), unsigned(p.h_kv * (p.group / NG)), unsigned(p.batch));
    hipLaunchKernelGGL((decode_split_kernel<D, NG>), grid, dim3(256), 0, stream, p);
    return hipGetLastError();
}

template <int D>
hipError_t launch_decode_d(const DecodeParams& p, hipStream_t stream) {
    hipError_t e;
    switch (p.heads_per_block) {
        case 1: e = launch_split<D, 1>(p, stream); break;
        case 2: e = launch_split<D, 2>(p, stream); break;
        case 3: e = launch_split<D, 3>(p, stream); break;
        case 4: e = launch_split<D, 4>(p, stream); break;
        case 5: e = launch_split<D, 5>(p, stream); break;
        case 6: e = launch_split<D, 6>(p, stream); break;
        case 7: e = launch_split<D, 7>(p, stream); break;
        case 8: e = launch_split<D, 8>(p, stream); break;
        default: return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(decode_merge_kernel<D>, dim3(unsigned(p.h_q), unsigned(p.batch)), dim3(D), 0,
                       stream, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_decode(const DecodeParams& p, int head_dim, hipStream_t stream) {
    if (p.splits < 1 || p.group % p.heads_per_block != 0) return hipErrorInvalidValue;
    if (int64_t(p.splits) * p.split_tokens < p.n_valid) return hipErrorInvalidValue;
    (void)hipGetLastError();
    return head_dim == 64 ? launch_decode_d<64>(p, stream) : launch_decode_d<128>(p, stream);
}

hipError_t launch_pack_kcache(const PackParams& p, int head_dim, hipStream_t stream) {
    const int64_t total = int64_t(p.batch) * p.n_k * p.h_kv * (head_dim / 16);
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    (void)hipGetLastError();
    if (head_dim == 64)
        hipLaunchKernelGGL(pack_kcache_kernel<64>, dim3(unsigned(blocks)), dim3(256), 0, stream, p);
    else
        hipLaunchKernelGGL(pack_kcache_kernel<128>, dim3(unsigned(blocks)), dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace atf
