// Windowed causal prefill for gfx950 (CDNA4): tiled attention with an online
// softmax in which the per-RoPE-wavelength window (Sec. 3.2 eq:window) is applied
// as a per-tile slice of the QK contraction axis (Sec. 3.3).
//
// Work decomposition
//   workgroup = 4 waves = 128 query rows of one (batch, query head); each wave owns
//   32 rows.  Key tiles of 64 keys are staged in LDS: K only for the pair-chunks
//   that some cell of the tile keeps, V in full and transposed.
//
// Matrix layout (v_mfma_f32_32x32x16_bf16, lane l, c = l % 32, h = l / 32)
//   S^T[key][row] = K[key][dims] * Q^T[dims][row]: A = K fragment (key c, dims
//   8h..8h+7 of the K-step), B = Q fragment (row c, same dims), so lane l ends up
//   holding query row c and keys 8*(v/4) + 4h + v%4 of a 32-key block (v < 16).
//   One query row per lane (per lane pair) makes the row max and row sum of the
//   softmax lane-local plus one cross-half exchange.
//   O^T[d][row] += V^T[d][key] * P^T[key][row]: the S^T registers, rounded to
//   bf16, are the B operand directly; V^T is read from the transposed LDS tile.
//
// Window as a K-slice (one K-step = one chunk of 8 rotary pairs = dims
// [8c, 8c+8) and [d/2 + 8c, d/2 + 8c + 8)).  For each (wave, 32-key block) the
// distances z of its cells span [zlo, zhi].  A chunk whose smallest threshold is
// >= zhi is kept whole (one MFMA); a chunk whose largest threshold is < zlo is
// skipped (neither loaded nor multiplied); otherwise the chunk is a boundary
// chunk: its pairs kept in every cell go into one MFMA with the other pairs'
// query dims zeroed, and each pair whose threshold falls inside [zlo, zhi) gets
// one MFMA of its own whose product is added only to the cells with z <= W_r.
// The result is exact per element: every cell sums exactly its kept pairs.
#include "atf_internal.hpp"

namespace atf {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr int kBM = kWaves * 32;  // query rows per workgroup
constexpr int kBN = 64;           // keys per tile
constexpr int kKPad = 8;          // bf16 padding per K row in LDS
constexpr int kVPad = 8;          // bf16 padding per transposed V row in LDS

template <int D>
struct Cfg {
    static constexpr int kHalf = D / 2;
    static constexpr int kChunks = D / 16;
    static constexpr int kKStride = D + kKPad;    // bf16 per K row
    static constexpr int kVStride = kBN + kVPad;  // bf16 per V^T row
};

__device__ __forceinline__ f32x16_t mfma(u32x4_t a, u32x4_t b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

// Keep only the pairs whose bit is set in `mask` (bit e = pair 8c+e of the
// chunk); a fragment holds the 8 dims of one half of the chunk, element e in
// dword e/2, low half for even e.
__device__ __forceinline__ u32x4_t keep_pairs(u32x4_t x, uint32_t mask) {
    u32x4_t r;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const uint32_t m = ((mask >> (2 * t)) & 1u ? 0x0000FFFFu : 0u) |
                           ((mask >> (2 * t + 1)) & 1u ? 0xFFFF0000u : 0u);
        r[t] = x[t] & m;
    }
    return r;
}

// Position of key k (0..63) inside a transposed V row: within every group of 16
// keys the order is [0-3, 8-11, 4-7, 12-15], so that lane half h finds the 8 keys
// it feeds to the PV MFMA (keys 4h..4h+3 and 8+4h..8+4h+3) contiguous.
__device__ __forceinline__ int vt_pos(int k) {
    return (k & ~12) | ((k & 4) << 1) | ((k & 8) >> 1);
}

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

template <int D>
__global__ __launch_bounds__(256, 2) void prefill_kernel(const PrefillParams p) {
    using C = Cfg<D>;
    __shared__ __attribute__((aligned(16))) uint16_t Ks[kBN * C::kKStride];
    __shared__ __attribute__((aligned(16))) uint16_t Vt[D * C::kVStride];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col = lane & 31;
    const int hh = lane >> 5;

    // heavy (late, long) query tiles are dispatched first; the heads of one
    // KV group are adjacent
    const int per_tile = p.h_q * p.batch;
    const int bid = blockIdx.x;
    const int qt = p.n_qtiles - 1 - bid / per_tile;
    const int rem = bid % per_tile;
    const int hq = rem % p.h_q;
    const int b = rem / p.h_q;
    const int g = hq / p.group;

    const int i0 = qt * kBM;
    const int tile_rows = min(kBM, p.n_q - i0);
    const int pos_first = p.q_pos0 + i0;
    const int pos_last = pos_first + tile_rows - 1;
    const int key_end = min(p.n_k, pos_last + 1);

    const int wrow0 = i0 + wave * 32;
    const int wrows = min(32, p.n_q - wrow0);  // rows of this wave (may be <= 0)
    const int wpos0 = p.q_pos0 + wrow0;
    const int wpos_last = wpos0 + wrows - 1;
    const int my_row = wrow0 + col;
    const int my_pos = wpos0 + col;
    const bool row_ok = col < wrows;

    const int64_t kv_row_stride = int64_t(p.h_kv) * D;
    const uint16_t* kbase = p.k + (int64_t(b) * p.n_k * p.h_kv + g) * D;
    const uint16_t* vbase = p.v + (int64_t(b) * p.n_k * p.h_kv + g) * D;

    // query fragments (B operand): row `col`, dims of half hh of every chunk
    u32x4_t qf[C::kChunks];
    {
        const uint16_t* qrow =
            p.q + ((int64_t(b) * p.n_q + my_row) * p.h_q + hq) * D + hh * C::kHalf;
#pragma unroll
        for (int c = 0; c < C::kChunks; ++c) {
            u32x4_t z = {0u, 0u, 0u, 0u};
            qf[c] = row_ok ? *reinterpret_cast<const u32x4_t*>(qrow + 8 * c) : z;
        }
    }

    f32x16_t oacc[D / 32];
#pragma unroll
    for (int i = 0; i < D / 32; ++i)
#pragma unroll
        for (int v = 0; v < 16; ++v) oacc[i][v] = 0.f;
    float m_run = -INFINITY;  // running row max, log2 domain (score * scale * log2 e)
    float l_run = 0.f;        // running normaliser (this lane's keys only)

    const bool wave_active = wrows > 0;

    for (int j0 = 0; j0 < key_end; j0 += kBN) {
        // chunks some cell of this workgroup tile keeps
        const int zlo_tile = max(0, pos_first - (j0 + kBN - 1));
        uint32_t need = 0;
#pragma unroll
        for (int c = 0; c < C::kChunks; ++c)
            if (p.win.chunk_max[c] >= zlo_tile) need |= 1u << c;

        __syncthreads();  // previous tile fully consumed
        // K tile: (key, 16-byte segment); segment s covers dims 8*(s % chunks) of half s / chunks
        for (int s = tid; s < kBN * 2 * C::kChunks; s += 256) {
            const int key = s / (2 * C::kChunks);
            const int seg = s % (2 * C::kChunks);
            const int c = seg % C::kChunks;
            const int half = seg / C::kChunks;
            if (!((need >> c) & 1u)) continue;
            const int j = j0 + key;
            const int off = half * C::kHalf + 8 * c;
            u32x4_t val = {0u, 0u, 0u, 0u};
            if (j < p.n_k) val = *reinterpret_cast<const u32x4_t*>(kbase + int64_t(j) * kv_row_stride + off);
            *reinterpret_cast<u32x4_t*>(&Ks[key * C::kKStride + off]) = val;
        }
        // V tile, transposed: (key pair, 16-byte segment), key pairs fastest so that
        // a wave's LDS stores hit consecutive dwords
        for (int s = tid; s < (kBN / 2) * (D / 8); s += 256) {
            const int kp = s % (kBN / 2);
            const int seg = s / (kBN / 2);
            const int j = j0 + 2 * kp;
            u32x4_t a = {0u, 0u, 0u, 0u}, c2 = {0u, 0u, 0u, 0u};
            if (j < p.n_k) a = *reinterpret_cast<const u32x4_t*>(vbase + int64_t(j) * kv_row_stride + 8 * seg);
            if (j + 1 < p.n_k)
                c2 = *reinterpret_cast<const u32x4_t*>(vbase + int64_t(j + 1) * kv_row_stride + 8 * seg);
            const int pos = vt_pos(2 * kp);
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const uint32_t lo = (a[t] & 0xFFFFu) | (c2[t] << 16);
                const uint32_t hi = (a[t] >> 16) | (c2[t] & 0xFFFF0000u);
                *reinterpret_cast<uint32_t*>(&Vt[(8 * seg + 2 * t) * C::kVStride + pos]) = lo;
                *reinterpret_cast<uint32_t*>(&Vt[(8 * seg + 2 * t + 1) * C::kVStride + pos]) = hi;
            }
        }
        __syncthreads();

        if (!wave_active || wpos_last < j0) continue;  // no row of this wave sees the tile

        f32x16_t sacc[2];
        bool blk_live[2];
#pragma unroll
        for (int b2 = 0; b2 < 2; ++b2) {
#pragma unroll
            for (int v = 0; v < 16; ++v) sacc[b2][v] = 0.f;
            const int jb = j0 + 32 * b2;
            const int zhi = wpos_last - jb;  // largest distance in the block
            blk_live[b2] = zhi >= 0 && jb < p.n_k;
            if (!blk_live[b2]) continue;
            const int zlo_raw = wpos0 - (jb + 31);
            const int zlo = max(0, zlo_raw);
            const uint16_t* krow = Ks + (32 * b2 + col) * C::kKStride + hh * C::kHalf;
            const int zbase = my_pos - jb - 4 * hh;  // z of register v is zbase - off(v)
#pragma unroll
            for (int c = 0; c < C::kChunks; ++c) {
                const int cmin = p.win.chunk_min[c];
                const int cmax = p.win.chunk_max[c];
                if (cmax < zlo) continue;  // no cell of the block keeps any pair of the chunk
                const u32x4_t kf = *reinterpret_cast<const u32x4_t*>(krow + 8 * c);
                if (cmin >= zhi) {  // every cell keeps every pair of the chunk
                    sacc[b2] = mfma(kf, qf[c], sacc[b2]);
                    continue;
                }
                uint32_t full = 0, part = 0;
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const int w = p.win.W[8 * c + e];
                    if (w >= zhi) full |= 1u << e;
                    else if (w >= zlo) part |= 1u << e;
                }
                if (full) sacc[b2] = mfma(kf, keep_pairs(qf[c], full), sacc[b2]);
                while (part) {
                    const int e = __builtin_ctz(part);
                    part &= part - 1;
                    f32x16_t zero;
#pragma unroll
                    for (int v = 0; v < 16; ++v) zero[v] = 0.f;
                    const f32x16_t t = mfma(kf, keep_pairs(qf[c], 1u << e), zero);
                    const int thr = zbase - p.win.W[8 * c + e];  // keep iff off(v) >= thr
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int off = 8 * (v / 4) + (v % 4);
                        sacc[b2][v] += off >= thr ? t[v] : 0.f;
                    }
                }
            }
            // causal mask and key bound (only blocks that reach the diagonal or n_k)
            if (zlo_raw < 0 || jb + 32 > p.n_k) {
                const int kbound = p.n_k - jb - 4 * hh;
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int off = 8 * (v / 4) + (v % 4);
                    if (off > zbase || off >= kbound) sacc[b2][v] = -INFINITY;
                }
            }
        }

        // online softmax (lane = query row; the two lane halves hold disjoint keys)
        float mx = -INFINITY;
#pragma unroll
        for (int b2 = 0; b2 < 2; ++b2)
            if (blk_live[b2])
#pragma unroll
                for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[b2][v]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run, mx * p.scale_log2);
        const float m_use = m_new == -INFINITY ? 0.f : m_new;
        const float alpha = exp2_fast(m_run - m_use);
        m_run = m_new;
        l_run *= alpha;
#pragma unroll
        for (int i = 0; i < D / 32; ++i)
#pragma unroll
            for (int v = 0; v < 16; ++v) oacc[i][v] *= alpha;

#pragma unroll
        for (int b2 = 0; b2 < 2; ++b2) {
            if (!blk_live[b2]) continue;
            float pr[16];
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                pr[v] = exp2_fast(__builtin_fmaf(sacc[b2][v], p.scale_log2, -m_use));
                l_run += pr[v];
            }
#pragma unroll
            for (int ks = 0; ks < 2; ++ks) {
                u32x4_t pb;
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
                    bf16x2_t two;
                    two[0] = (__bf16)pr[8 * ks + 2 * t];
                    two[1] = (__bf16)pr[8 * ks + 2 * t + 1];
                    pb[t] = __builtin_bit_cast(uint32_t, two);
                }
                const uint16_t* vrow = Vt + col * C::kVStride + 32 * b2 + 16 * ks + 8 * hh;
#pragma unroll
                for (int i = 0; i < D / 32; ++i) {
                    const u32x4_t vf =
                        *reinterpret_cast<const u32x4_t*>(vrow + 32 * i * C::kVStride);
                    oacc[i] = mfma(vf, pb, oacc[i]);
                }
            }
        }
    }

    if (!wave_active) return;
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    if (!row_ok) return;
    const float inv = 1.0f / l_tot;
    uint16_t* orow = p.o + ((int64_t(b) * p.n_q + my_row) * p.h_q + hq) * D;
#pragma unroll
    for (int i = 0; i < D / 32; ++i) {
#pragma unroll
        for (int grp = 0; grp < 4; ++grp) {
            typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
            bf16x4_t out;
#pragma unroll
            for (int t = 0; t < 4; ++t) out[t] = (__bf16)(oacc[i][4 * grp + t] * inv);
            *reinterpret_cast<bf16x4_t*>(orow + 32 * i + 8 * grp + 4 * hh) = out;
        }
    }
    if (hh == 0)
        p.lse[(int64_t(b) * p.h_q + hq) * p.n_q + my_row] =
            m_run * 0.69314718055994531f + logf(l_tot);
}

}  // namespace

hipError_t launch_prefill(const PrefillParams& p_in, int head_dim, hipStream_t stream) {
    PrefillParams p = p_in;
    p.n_qtiles = (p.n_q + kBM - 1) / kBM;
    const int64_t blocks = int64_t(p.n_qtiles) * p.h_q * p.batch;
    if (blocks <= 0 || blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
    (void)hipGetLastError();
    if (head_dim == 64)
        hipLaunchKernelGGL(prefill_kernel<64>, dim3(unsigned(blocks)), dim3(256), 0, stream, p);
    else
        hipLaunchKernelGGL(prefill_kernel<128>, dim3(unsigned(blocks)), dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace atf
