// Windowed causal prefill for gfx950 (CDNA4): tiled attention with an online
// softmax in which the per-RoPE-wavelength window (Sec. 3.2 eq:window) is applied
// as a per-tile slice of the QK contraction axis (Sec. 3.3).
//
// Work decomposition
//   A workgroup of 8 waves owns 256 query rows that share one KV head: P = 256/G
//   consecutive positions x the G query heads of the group (row f -> position
//   f / G, head f % G), so every K/V tile staged in LDS serves 256 rows.  Each
//   wave owns 32 rows (one MFMA row-block); two waves share a SIMD so one wave's
//   softmax (VALU) overlaps the other's matrix work.  Key tiles of 64 are
//   double-buffered in LDS and filled by global_load_lds_dwordx4 (global memory
//   straight into LDS, no register staging) one tile ahead of the compute.
//
// LDS layout: K and V tiles are row-major [key][d] with padded rows, chosen so
// that the K fragment reads (rows at one 16-byte segment) and the transposed V
// reads (4 rows x 32 bytes per 16 lanes) hit distinct banks while every fragment
// address is a per-lane base plus an immediate offset.
//
// Matrix layout (v_mfma_f32_32x32x16_bf16, lane l, c = l % 32, h = l / 32)
//   S^T[key][row] = K[key][dims] * Q^T[dims][row]: A = K fragment (key c, dims
//   8h..8h+7 of the K-step), B = Q fragment (row c, same dims), so lane l holds
//   query row c and keys 8*(v/4) + 4h + v%4 of a 32-key block (v < 16).  One query
//   row per lane pair makes the row max and sum lane-local plus one exchange.
//   O^T[d][row] += V^T[d][key] * P^T[key][row]: the S^T registers, rounded to
//   bf16, are the B operand as they are; the V^T operand is read from the
//   row-major V tile with ds_read_b64_tr_b16 (within 16 lanes, a transposed read:
//   lane i gets column d0 + i of four consecutive key rows).
//
// Window as a K-slice (one K-step = one chunk of 8 rotary pairs = dims
// [8c, 8c+8) and [d/2 + 8c, d/2 + 8c + 8)).  For each (wave, 32-key block) the
// distances z of its cells span [zlo, zhi].  A chunk whose smallest threshold is
// >= zhi is kept whole (one MFMA); a chunk whose largest threshold is < zlo is
// skipped (not loaded into LDS when the whole tile skips it, never multiplied);
// otherwise the chunk is a boundary chunk: its pairs kept in every cell go into
// one MFMA with the other pairs' query dims zeroed, and each pair whose threshold
// falls inside [zlo, zhi) gets one MFMA of its own whose product is added only
// to the cells with z <= W_r.  Every cell sums exactly its kept pairs.  With the
// window off (no threshold below the largest distance) the kernel is compiled
// without any of this: every chunk is a full K-step.
//
// Softmax: fp32 in the log2 domain.  The running max is raised only when a row's
// tile max exceeds it by more than kRescale (log2 units); otherwise the stale
// max is kept, probabilities are at most 2^kRescale, and the output and
// normaliser need no rescaling -- the result is the same softmax.  Row sums add
// the fp32 probabilities; the PV MFMA consumes them rounded to bf16.
#include "atf_internal.hpp"

namespace atf {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef short s16x8_t __attribute__((ext_vector_type(8)));

constexpr int kWaves = 8;
constexpr int kThreads = kWaves * 64;
constexpr int kRows = kWaves * 32;  // query rows per workgroup
constexpr int kBN = 64;             // keys per tile
constexpr float kRescale = 8.0f;    // lazy-rescale threshold, log2 units

// Row strides: K rows carry 16 bytes of padding, so 8 consecutive rows read at
// one 16-byte segment fall on distinct banks; V rows are a multiple of 128 bytes
// plus 64, so the four rows one transposed read touches start 64 bytes apart
// modulo the 256-byte bank line.  Both tiles are whole kilobytes: a wave-wide
// 16-byte direct load fills 1 KB of a tile, slot s = 64 * load + lane holding
// (row s / slots-per-row, segment s % slots-per-row); slots past a row's data
// are padding and receive a dummy load.
template <int D>
struct Cfg {
    static constexpr int kHalf = D / 2;
    static constexpr int kChunks = D / 16;
    static constexpr int kSegs = D / 8;          // 16-byte data segments per row
    static constexpr int kKStride = D + 8;       // bf16 per K row in LDS
    static constexpr int kVStride = D + 32;      // bf16 per V row in LDS
    static constexpr int kKSlots = kKStride / 8;
    static constexpr int kVSlots = kVStride / 8;
    static constexpr int kKTile = kBN * kKStride;  // bf16
    static constexpr int kVTile = kBN * kVStride;
    static constexpr int kKLoads = kKTile / 512;   // wave-wide loads per tile
    static constexpr int kVLoads = kVTile / 512;
    static_assert(kKTile % 512 == 0 && kVTile % 512 == 0, "tiles must be whole kilobytes");
};

__device__ __forceinline__ f32x16_t mfma(u32x4_t a, u32x4_t b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                   __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
}

__device__ __forceinline__ f32x16_t zero16() {
    f32x16_t z;
#pragma unroll
    for (int v = 0; v < 16; ++v) z[v] = 0.f;
    return z;
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

__device__ __forceinline__ float exp2_fast(float x) { return __builtin_amdgcn_exp2f(x); }

typedef __attribute__((address_space(3))) char lds_char;

// Transposed 4x4-block read of 16-bit elements from LDS (ds_read_b64_tr_b16).
__device__ __forceinline__ s16x4_t lds_read_tr(const uint16_t* p) {
    typedef __attribute__((address_space(3))) s16x4_t lds_s16x4;
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)((lds_char*)(p)));
}

// 16 bytes per lane from global memory straight into LDS at lds_wave + 16 * lane
// (lds_wave must be the same for every lane of the wave).
__device__ __forceinline__ void load_to_lds(const uint16_t* g, uint16_t* lds_wave) {
    __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)((lds_char*)lds_wave),
                                     16, 0, 0);
}

template <int D, bool kWin>
__global__ __launch_bounds__(kThreads, D == 64 ? 4 : 2) void prefill_kernel(const PrefillParams p) {
    using C = Cfg<D>;
    __shared__ __attribute__((aligned(16))) uint16_t Ks[2][C::kKTile];
    __shared__ __attribute__((aligned(16))) uint16_t Vs[2][C::kVTile];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col = lane & 31;
    const int hh = lane >> 5;

    // block -> (position tile, kv head, batch); heavy (late) tiles first.  Blocks
    // are dealt to the 8 XCDs round-robin, so with h_kv * batch a multiple or a
    // divisor of 8 every XCD keeps to fixed KV heads and its L2 serves them.
    const int per_tile = p.h_kv * p.batch;
    const int bid = blockIdx.x;
    const int qt = p.n_qtiles - 1 - bid / per_tile;
    const int rem = bid % per_tile;
    const int g = rem % p.h_kv;
    const int b = rem / p.h_kv;
    const int G = p.group;

    const int i0 = qt * p.pos_per_tile;  // first query row (position index)
    const int npos = min(p.pos_per_tile, p.n_q - i0);
    const int rows_valid = npos * G;
    const int pos_first = p.q_pos0 + i0;
    const int pos_last = pos_first + npos - 1;
    const int key_end = min(p.n_k, pos_last + 1);

    // this lane's row: workgroup row 32 * wave + col
    const int f = 32 * wave + col;
    const bool row_ok = f < rows_valid;
    const int ff = row_ok ? f : 0;
    const int my_qrow = i0 + ff / G;
    const int my_head = g * G + ff % G;
    const int my_pos = p.q_pos0 + my_qrow;
    const int wf0 = 32 * wave;
    const bool wave_active = wf0 < rows_valid;
    const int wf1 = min(wf0 + 31, rows_valid - 1);
    const int wp_min = pos_first + wf0 / G;
    const int wp_max = pos_first + (wave_active ? wf1 : wf0) / G;
    // lane r holds the threshold of pair r (pairs past d/2 never count)
    const int my_w = lane < C::kHalf ? p.win.W[lane] : -1;

    const int64_t kv_row_stride = int64_t(p.h_kv) * D;
    const uint16_t* kbase = p.k + (int64_t(b) * p.n_k * p.h_kv + g) * D;
    const uint16_t* vbase = p.v + (int64_t(b) * p.n_k * p.h_kv + g) * D;

    // query fragments (B operand): row `col`, dims of half hh of every chunk
    u32x4_t qf[C::kChunks];
    {
        const uint16_t* qrow =
            p.q + ((int64_t(b) * p.n_q + my_qrow) * p.h_q + my_head) * D + hh * C::kHalf;
#pragma unroll
        for (int c = 0; c < C::kChunks; ++c) {
            u32x4_t z = {0u, 0u, 0u, 0u};
            if (row_ok) z = *reinterpret_cast<const u32x4_t*>(qrow + 8 * c);
            qf[c] = z;
        }
    }

    // chunks that some cell of the workgroup tile at keys [j0, j0 + 64) keeps, plus
    // the last chunk: the first QK MFMA of a block always multiplies it (with the
    // query dims of unkept pairs zeroed), so it must hold finite data
    auto tile_need = [&](int j0) -> uint32_t {
        if (!kWin) return (1u << C::kChunks) - 1u;
        const int zlo = max(0, pos_first - (j0 + kBN - 1));
        uint32_t need = 1u << (C::kChunks - 1);
#pragma unroll
        for (int c = 0; c < C::kChunks; ++c)
            if (p.win.chunk_max[c] >= zlo) need |= 1u << c;
        return need;
    };
    // issue the global -> LDS loads of the tile at key j0 into buffer `buf`; wave w
    // issues the tile's wave-wide loads w, w + 8, ...  A lane's (row, segment) slot
    // in each load is fixed, so its element offset within the tile is computed once;
    // the tile base is wave-uniform.  In a tile that crosses n_k, rows past n_k
    // re-read the last key (finite values; their scores are masked).
    constexpr int kKPer = (C::kKLoads + kWaves - 1) / kWaves;
    constexpr int kVPer = (C::kVLoads + kWaves - 1) / kWaves;
    int k_row[kKPer], k_seg[kKPer], v_row_l[kVPer], v_seg[kVPer];
#pragma unroll
    for (int t = 0; t < kKPer; ++t) {
        const int s = 64 * (wave + kWaves * t) + lane;
        k_row[t] = s / C::kKSlots;
        const int seg = s % C::kKSlots;
        k_seg[t] = seg < C::kSegs ? seg : -1;  // -1: padding slot
    }
#pragma unroll
    for (int t = 0; t < kVPer; ++t) {
        const int s = 64 * (wave + kWaves * t) + lane;
        v_row_l[t] = s / C::kVSlots;
        const int seg = s % C::kVSlots;
        v_seg[t] = seg < C::kSegs ? seg : 0;  // padding slots load a dummy
    }
    auto issue = [&](int j0, int buf) {
        const uint32_t need = tile_need(j0);
        const bool tail = j0 + kBN > p.n_k;
        const uint16_t* kt = kbase + int64_t(j0) * kv_row_stride;
        const uint16_t* vt = vbase + int64_t(j0) * kv_row_stride;
        const int last = p.n_k - 1 - j0;  // last valid row of the tile
#pragma unroll
        for (int t = 0; t < kKPer; ++t) {
            const int u = wave + kWaves * t;
            if (u >= C::kKLoads) break;
            const int seg = k_seg[t];
            const int r = tail ? min(k_row[t], last) : k_row[t];
            if (seg < 0 || ((need >> (seg % C::kChunks)) & 1u))
                load_to_lds(kt + r * int(kv_row_stride) + 8 * (seg < 0 ? 0 : seg), &Ks[buf][512 * u]);
        }
#pragma unroll
        for (int t = 0; t < kVPer; ++t) {
            const int u = wave + kWaves * t;
            if (u >= C::kVLoads) break;
            const int r = tail ? min(v_row_l[t], last) : v_row_l[t];
            load_to_lds(vt + r * int(kv_row_stride) + 8 * v_seg[t], &Vs[buf][512 * u]);
        }
    };

    // per-lane LDS fragment bases (buffer 0); fragment reads add immediate offsets
    const int k_off[2] = {col * C::kKStride + hh * C::kHalf,
                          (32 + col) * C::kKStride + hh * C::kHalf};
    const int v_dsub = 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
    const int v_row = 4 * hh + ((lane & 15) >> 2);

    f32x16_t oacc[D / 32];
#pragma unroll
    for (int i = 0; i < D / 32; ++i) oacc[i] = zero16();
    float m_run = -INFINITY;  // running (possibly stale) max, log2 domain
    float l_run = 0.f;        // normaliser over this lane's keys
    const float sc = p.scale_log2;

    issue(0, 0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();

    int buf = 0;
    for (int j0 = 0; j0 < key_end; j0 += kBN, buf ^= 1) {
        const bool has_next = j0 + kBN < key_end;
        if (has_next) issue(j0 + kBN, buf ^ 1);

        if (wave_active && wp_max >= j0) {
            const uint16_t* Kb = Ks[buf];
            const uint16_t* Vb = Vs[buf];
            // ---- QK for both 32-key blocks of the tile (the matrix phase; the window's
            // branches live here).  Block 0 always has a causal key; block 1 may not.
            const bool live1 = wp_max >= j0 + 32 && j0 + 32 < p.n_k;
            f32x16_t sacc[2];
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                if (kb == 1 && !live1) {
                    sacc[1] = zero16();  // masked below
                    continue;
                }
                const int jb = j0 + 32 * kb;
                const int zhi = wp_max - jb;
                const int zlo = max(0, wp_min - (jb + 31));
                // every K fragment of the block is read before any branch so that the
                // reads overlap; a chunk the block does not keep is never multiplied
                const uint16_t* krow = Kb + k_off[kb];
                u32x4_t kf[C::kChunks];
#pragma unroll
                for (int c = 0; c < C::kChunks; ++c)
                    kf[c] = *reinterpret_cast<const u32x4_t*>(krow + 8 * c);
                f32x16_t acc;
                if (!kWin) {
                    acc = mfma(kf[C::kChunks - 1], qf[C::kChunks - 1], zero16());
#pragma unroll
                    for (int c = C::kChunks - 2; c >= 0; --c) acc = mfma(kf[c], qf[c], acc);
                } else {
                    // all pairs classified at once: lane r holds W_r; bit r of `full` = pair r
                    // kept in every cell of the block, of `keep` = kept in some cell
                    const uint64_t full = __ballot(my_w >= zhi);
                    const uint64_t keep = __ballot(my_w >= zlo);
                    // lowest frequencies (largest windows) first: the first MFMA always runs
                    // (pairs no cell keeps zeroed) and starts from a zero accumulator.  Each
                    // chunk has one MFMA site, so the scores are updated in place.
#pragma unroll
                    for (int c = C::kChunks - 1; c >= 0; --c) {
                        const uint32_t fc = uint32_t(full >> (8 * c)) & 0xFFu;
                        if (c == C::kChunks - 1) {
                            acc = mfma(kf[c], keep_pairs(qf[c], fc), zero16());
                        } else if (fc) {
                            u32x4_t qb = qf[c];
                            if (fc != 0xFFu) qb = keep_pairs(qb, fc);
                            acc = mfma(kf[c], qb, acc);
                        }
                    }
                    // pairs whose window ends inside the block: one MFMA each, added where
                    // z <= W_r (register v holds distance zbase - off(v): keep iff off(v) >= thr)
                    uint64_t part = keep & ~full;
                    while (part) {
                        const int r = __builtin_ctzll(part);
                        part &= part - 1;
                        const int c = r >> 3;
                        u32x4_t kfc = kf[0], qfc = qf[0];
#pragma unroll
                        for (int cc = 1; cc < C::kChunks; ++cc)
                            if (cc == c) {
                                kfc = kf[cc];
                                qfc = qf[cc];
                            }
                        const f32x16_t t = mfma(kfc, keep_pairs(qfc, 1u << (r & 7)), zero16());
                        const int thr = my_pos - jb - 4 * hh - p.win.W[r];
#pragma unroll
                        for (int v = 0; v < 16; ++v) {
                            const int off = 8 * (v / 4) + (v % 4);
                            acc[v] += off >= thr ? t[v] : 0.f;
                        }
                    }
                }
                sacc[kb] = acc;
            }
            // ---- causal mask and key bound, only in tiles that reach the diagonal or n_k
            if (wp_min - (j0 + kBN - 1) < 0 || j0 + kBN > p.n_k) {
#pragma unroll
                for (int kb = 0; kb < 2; ++kb) {
                    const int jb = j0 + 32 * kb;
                    const int kbound = p.n_k - jb - 4 * hh;
                    const int zbase = my_pos - jb - 4 * hh;
#pragma unroll
                    for (int v = 0; v < 16; ++v) {
                        const int off = 8 * (v / 4) + (v % 4);
                        if (off > zbase || off >= kbound) sacc[kb][v] = -INFINITY;
                    }
                }
            }
            // ---- online softmax over the tile (lane = query row; the two lane halves
            // hold disjoint keys).  One rescale check per tile; below it the softmax and
            // the PV products of both blocks are branch-free, so the PV matrix work of
            // block 0 overlaps the exponentials of block 1.
            float mx = -INFINITY;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb)
#pragma unroll
                for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[kb][v]);
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float cand = mx * sc;
            if (__any(cand > m_run + kRescale)) {
                const float m_new = fmaxf(m_run, cand);
                const float alpha = exp2_fast(m_run - (m_new == -INFINITY ? 0.f : m_new));
                m_run = m_new;
                l_run *= alpha;
#pragma unroll
                for (int i = 0; i < D / 32; ++i)
#pragma unroll
                    for (int v = 0; v < 16; ++v) oacc[i][v] *= alpha;
            }
            const float m_use = m_run == -INFINITY ? 0.f : m_run;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                u32x4_t pb[2];
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        const float a = exp2_fast(__builtin_fmaf(sacc[kb][8 * ks + 2 * t], sc, -m_use));
                        const float c2 = exp2_fast(__builtin_fmaf(sacc[kb][8 * ks + 2 * t + 1], sc, -m_use));
                        l_run += a;
                        l_run += c2;
                        bf16x2_t two;
                        two[0] = (__bf16)a;
                        two[1] = (__bf16)c2;
                        pb[ks][t] = __builtin_bit_cast(uint32_t, two);
                    }
                }
                // PV: V^T fragments by transposed LDS reads.  Lane group of 16: key rows
                // 4 * hh + (l % 16) / 4 (8 rows further for elements 4..7), dims
                // 16 * ((l / 16) % 2) + 4 * (l % 4) of each 32-dim block.
#pragma unroll
                for (int ks = 0; ks < 2; ++ks) {
                    const uint16_t* vp = Vb + (32 * kb + 16 * ks + v_row) * C::kVStride + v_dsub;
#pragma unroll
                    for (int i = 0; i < D / 32; ++i) {
                        const s16x4_t lo = lds_read_tr(vp + 32 * i);
                        const s16x4_t hi = lds_read_tr(vp + 8 * C::kVStride + 32 * i);
                        const s16x8_t both = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
                        oacc[i] = mfma(__builtin_bit_cast(u32x4_t, both), pb[ks], oacc[i]);
                    }
                }
            }
        }

        __builtin_amdgcn_s_waitcnt(0);  // this thread's loads of the next tile have landed
        __syncthreads();
    }

    if (!wave_active) return;
    const float l_tot = l_run + __shfl_xor(l_run, 32);
    if (!row_ok) return;
    const float inv = 1.0f / l_tot;
    uint16_t* orow = p.o + ((int64_t(b) * p.n_q + my_qrow) * p.h_q + my_head) * D;
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
        p.lse[(int64_t(b) * p.h_q + my_head) * p.n_q + my_qrow] =
            m_run * 0.69314718055994531f + logf(l_tot);
}

template <int D>
hipError_t launch_d(const PrefillParams& p, unsigned blocks, bool window_on, hipStream_t stream) {
    if (window_on)
        hipLaunchKernelGGL((prefill_kernel<D, true>), dim3(blocks), dim3(kThreads), 0, stream, p);
    else
        hipLaunchKernelGGL((prefill_kernel<D, false>), dim3(blocks), dim3(kThreads), 0, stream, p);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_prefill(const PrefillParams& p_in, int head_dim, hipStream_t stream) {
    PrefillParams p = p_in;
    if (p.group < 1 || p.group > kRows) return hipErrorInvalidValue;
    p.pos_per_tile = kRows / p.group;
    p.n_qtiles = (p.n_q + p.pos_per_tile - 1) / p.pos_per_tile;
    const int64_t blocks = int64_t(p.n_qtiles) * p.h_kv * p.batch;
    if (blocks <= 0 || blocks > 0x7fffffff) return hipErrorInvalidConfiguration;
    // the window is off when no threshold is below the largest possible distance
    const int64_t max_dist = int64_t(p.q_pos0) + p.n_q - 1;
    bool window_on = false;
    for (int r = 0; r < head_dim / 2; ++r)
        if (int64_t(p.win.W[r]) < max_dist) window_on = true;
    (void)hipGetLastError();
    return head_dim == 64 ? launch_d<64>(p, unsigned(blocks), window_on, stream)
                          : launch_d<128>(p, unsigned(blocks), window_on, stream);
}

}  // namespace atf
