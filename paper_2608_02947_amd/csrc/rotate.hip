// RoPE at write time (App. B sets it against rotating at read time): the keys of an
// unrotated K cache turned once, each to its own position, into a second cache or in
// place, and the same rotation fused into the cache append; the pre-rotated prefill and
// decode then read the result.  It costs one read and one write of the keys and every
// (key, pair) rotation, whatever the window keeps, and a rotated copy's memory; a long
// prefill over an unrotated cache can take it instead of the read-time path when that
// memory is at hand.
//
// Memory-bound.  One thread per (key, pair-chunk): the chunk's 32 bytes (the first
// components of its 8 pairs, then the second) are read as two 16-byte loads, the 8
// angles evaluated directly (0.64 fixed-point fraction, v_cos_f32 / v_sin_f32 in
// revolutions), rotated in fp32 and rounded to bf16.  Whole cache: grid y = the
// (batch, kv head, chunk) stream, x over its tokens, so a block's chunk and its 8
// frequencies are uniform and consecutive threads touch consecutive 32-byte records.

#include "atf_internal.hpp"
#include "rope.hpp"

namespace atf {
namespace {

template <int D>
__global__ __launch_bounds__(256) void rotate_kcache_kernel(const RotateParams p) {
    constexpr int kChunks = D / 16;
    const int stream = blockIdx.y;  // (b * h_kv + g) * kChunks + c
    const int c = stream % kChunks;
    const int64_t off = int64_t(stream) * p.cache_tokens * 16;
    const uint16_t* src = p.src + off;
    uint16_t* dst = p.dst + off;
    for (int64_t t = int64_t(blockIdx.x) * 256 + threadIdx.x; t < p.n_k;
         t += int64_t(gridDim.x) * 256) {
        const rope::u32x4_t x = *reinterpret_cast<const rope::u32x4_t*>(src + 16 * t);
        const rope::u32x4_t y = *reinterpret_cast<const rope::u32x4_t*>(src + 16 * t + 8);
        float cs8[8], sn8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float u = rope::revolutions(uint32_t(t), make_uint2(p.rope_rho_hi[8 * c + e],
                                                                      p.rope_rho_lo[8 * c + e]));
            cs8[e] = __builtin_amdgcn_cosf(u);
            sn8[e] = __builtin_amdgcn_sinf(u);
        }
        *reinterpret_cast<rope::u32x4_t*>(dst + 16 * t) = rope::rotate_cs(x, y, 0, cs8, sn8);
        *reinterpret_cast<rope::u32x4_t*>(dst + 16 * t + 8) = rope::rotate_cs(y, x, 1, cs8, sn8);
    }
}

// Append with RoPE: keys as the projections give them ([B][n_k][h_kv][d], unrotated),
// each turned to its cache position pos0 + t and written into the pair-chunk-major
// cache, one thread per (token, kv head, chunk) as atf_pack_kcache lays them out.
template <int D>
__global__ __launch_bounds__(256) void append_rotated_k_kernel(const RotateParams p) {
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
        const rope::u32x4_t x = *reinterpret_cast<const rope::u32x4_t*>(src + 8 * c);
        const rope::u32x4_t y = *reinterpret_cast<const rope::u32x4_t*>(src + D / 2 + 8 * c);
        const uint32_t pos = uint32_t(p.pos0 + t);
        float cs8[8], sn8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float u = rope::revolutions(pos, make_uint2(p.rope_rho_hi[8 * c + e],
                                                              p.rope_rho_lo[8 * c + e]));
            cs8[e] = __builtin_amdgcn_cosf(u);
            sn8[e] = __builtin_amdgcn_sinf(u);
        }
        uint16_t* dst = p.dst + (((int64_t(b) * p.h_kv + g) * kChunks + c) * p.cache_tokens + pos) * 16;
        *reinterpret_cast<rope::u32x4_t*>(dst) = rope::rotate_cs(x, y, 0, cs8, sn8);
        *reinterpret_cast<rope::u32x4_t*>(dst + 8) = rope::rotate_cs(y, x, 1, cs8, sn8);
    }
}

// The paged form: one thread per (token, kv head, chunk), the token's page from the
// row's block table (entries outside the pool are skipped); K rotated as above into the
// page's pair-chunk-major slot, and the two 8-dim pieces of V that share the chunk's
// dims (d0 = 8 c and d/2 + 8 c) copied into the page's 16-token block, slot 8 h + e for
// token 8 (e / 4) + 4 h + e % 4 of the block, as atf_cache_append_paged writes them.
template <int D>
__global__ __launch_bounds__(256) void append_paged_rotated_kernel(const RotatePagedParams rp) {
    constexpr int kChunks = D / 16;
    const AppendPagedParams& p = rp.a;
    const int64_t total = int64_t(p.batch) * p.n_new * p.h_kv * kChunks;
    for (int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x; idx < total;
         idx += int64_t(gridDim.x) * 256) {
        const int c = int(idx % kChunks);
        int64_t r = idx / kChunks;
        const int g = int(r % p.h_kv);
        r /= p.h_kv;
        const int t = int(r % p.n_new);
        const int b = int(r / p.n_new);
        const int pos = p.pos0 + t;
        const int page = p.block_table[int64_t(b) * p.max_pages + pos / p.page_tokens];
        if (page < 0 || page >= p.num_pages) continue;
        const int slot = pos % p.page_tokens;
        const int64_t src = ((int64_t(b) * p.n_new + t) * p.h_kv + g) * D;
        const rope::u32x4_t x = *reinterpret_cast<const rope::u32x4_t*>(p.k_src + src + 8 * c);
        const rope::u32x4_t y = *reinterpret_cast<const rope::u32x4_t*>(p.k_src + src + D / 2 + 8 * c);
        float cs8[8], sn8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const float u = rope::revolutions(uint32_t(pos), make_uint2(rp.rope_rho_hi[8 * c + e],
                                                                        rp.rope_rho_lo[8 * c + e]));
            cs8[e] = __builtin_amdgcn_cosf(u);
            sn8[e] = __builtin_amdgcn_sinf(u);
        }
        uint16_t* kd = p.k_pages + (((int64_t(page) * p.h_kv + g) * kChunks + c) * p.page_tokens + slot) * 16;
        *reinterpret_cast<rope::u32x4_t*>(kd) = rope::rotate_cs(x, y, 0, cs8, sn8);
        *reinterpret_cast<rope::u32x4_t*>(kd + 8) = rope::rotate_cs(y, x, 1, cs8, sn8);
        const int e16 = slot % 16;
        const int h = (e16 % 8) / 4, e = (e16 / 8) * 4 + e16 % 4;
        uint16_t* vd = p.v_pages + ((int64_t(page) * p.h_kv + g) * (p.page_tokens / 16) + slot / 16) *
                                       int64_t(D) * 16 + 8 * h + e;
#pragma unroll
        for (int half = 0; half < 2; ++half) {
            const int d0 = 8 * c + half * (D / 2);
#pragma unroll
            for (int q = 0; q < 8; ++q) vd[int64_t(d0 + q) * 16] = p.v_src[src + d0 + q];
        }
    }
}

}  // namespace

hipError_t launch_append_paged_rotated(const RotatePagedParams& p, int head_dim, hipStream_t stream) {
    const int64_t total = int64_t(p.a.batch) * p.a.n_new * p.a.h_kv * (head_dim / 16);
    if (total < 1) return hipErrorInvalidConfiguration;
    const int64_t blocks = (total + 255) / 256;
    const unsigned grid = unsigned(blocks < 16384 ? blocks : 16384);
    (void)hipGetLastError();
    if (head_dim == 64)
        hipLaunchKernelGGL(append_paged_rotated_kernel<64>, dim3(grid), dim3(256), 0, stream, p);
    else
        hipLaunchKernelGGL(append_paged_rotated_kernel<128>, dim3(grid), dim3(256), 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_append_rotated_k(const RotateParams& p, int head_dim, hipStream_t stream) {
    const int64_t total = int64_t(p.batch) * p.n_k * p.h_kv * (head_dim / 16);
    if (total < 1) return hipErrorInvalidConfiguration;
    const int64_t blocks = (total + 255) / 256;
    const unsigned grid = unsigned(blocks < 16384 ? blocks : 16384);
    (void)hipGetLastError();
    if (head_dim == 64)
        hipLaunchKernelGGL(append_rotated_k_kernel<64>, dim3(grid), dim3(256), 0, stream, p);
    else
        hipLaunchKernelGGL(append_rotated_k_kernel<128>, dim3(grid), dim3(256), 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_rotate_kcache(const RotateParams& p, int head_dim, hipStream_t stream) {
    const int64_t streams = int64_t(p.batch) * p.h_kv * (head_dim / 16);
    if (streams < 1 || streams > 65535 || p.n_k < 1) return hipErrorInvalidConfiguration;
    const int64_t xb = (int64_t(p.n_k) + 255) / 256;
    const dim3 grid(unsigned(xb < 1024 ? xb : 1024), unsigned(streams));
    (void)hipGetLastError();
    if (head_dim == 64)
        hipLaunchKernelGGL(rotate_kcache_kernel<64>, grid, dim3(256), 0, stream, p);
    else
        hipLaunchKernelGGL(rotate_kcache_kernel<128>, grid, dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace atf
