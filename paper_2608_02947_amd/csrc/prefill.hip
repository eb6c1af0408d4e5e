// Windowed causal prefill for gfx950 (CDNA4): tiled attention with an online
// softmax in which the per-RoPE-wavelength window (Sec. 3.2 eq:window) is applied
// as a per-tile slice of the QK contraction axis (Sec. 3.3).
//
// Work decomposition
//   A workgroup of W waves owns 32 W query rows that share one KV head: P = 32W/G
//   consecutive positions x the G query heads of the group (row f -> position
//   f / G, head f % G), so every K/V tile staged in LDS serves all of them.  Each
//   wave owns 32 rows (one MFMA row-block).  W = 8 at d = 128 (two waves per
//   SIMD), W = 4 at d = 64 (three workgroups per CU).  Key tiles of 64 rotate
//   through LDS buffers filled by global_load_lds_dwordx4 (global memory straight
//   into LDS, no register staging) one tile ahead of the compute.
//
// K comes from the pair-chunk-major cache (the decode layout): chunk c of a KV
// head is a stream of 32 bytes per key (dims [8c, 8c+8) then [d/2+8c, d/2+8c+8)),
// so one wave-wide direct load fetches one chunk of 32 keys as 1 KB of contiguous
// memory, and a chunk that no cell of the tile keeps is skipped by one
// wave-uniform branch -- its bytes are never read from HBM.  In LDS the K tile is
// [chunk][32-key block][half][key][8 bf16]: a fragment read of 64 lanes covers
// 1 KB without bank conflicts.  V also comes from the decode cache: 16-token
// blocks stored [d][16 slots], slot 8h + e holding token 8(e/4) + 4h + e%4 of the
// block.  A 64-key tile is four consecutive blocks, one contiguous copy into LDS,
// and the 8 slots a lane needs for the PV operand are 16 contiguous bytes.
//
// Matrix layout (v_mfma_f32_32x32x16_bf16, lane l, c = l % 32, h = l / 32)
//   S^T[key][row] = K[key][dims] * Q^T[dims][row]: A = K fragment (key c, dims
//   8h..8h+7 of the K-step), B = Q fragment (row c, same dims), so lane l holds
//   query row c and keys 8*(v/4) + 4h + v%4 of a 32-key block (v < 16).  One query
//   row per lane pair makes the row max and sum lane-local plus one exchange.
//   O^T[d][row] += V^T[d][key] * P^T[key][row]: the S^T registers, rounded to
//   bf16, are the B operand as they are (element e of lane half h = key
//   8(e/4) + 4h + e%4 of a 16-key group); the V^T operand of lane (dim c, half h)
//   is slots 8h .. 8h+7 of dim row c of the packed block: the same keys.
//
// Window as a K-slice (one K-step = one chunk of 8 rotary pairs = dims
// [8c, 8c+8) and [d/2 + 8c, d/2 + 8c + 8)).  Whether pair r contributes to a cell
// depends only on the cell's distance z (keep iff z <= W_r).
//   Uniform tiles.  When no threshold falls inside the distance range of a wave's
//   tile, every pair is either kept in all of its cells or in none.  With
//   thresholds non-decreasing in r, the kept pairs are a suffix r >= rf, so the
//   tile's QK is the chunks above rf / 8 in full plus chunk rf / 8 with the query
//   dims of the pairs below rf zeroed.  That set stays the same for a run of
//   consecutive tiles (until the next threshold enters the distance range), and
//   each wave runs such a run in a loop compiled for its chunk count: straight
//   matrix code with no per-tile branch.
//   Other tiles (a threshold inside the range, or a table that is not monotone)
//   take the general path: per 32-key block, two ballots classify all pairs at
//   once (kept in every cell / in some cell); whole chunks go into one MFMA each
//   with the query dims of pairs kept nowhere zeroed, and each pair whose
//   threshold lies inside the block's range gets one MFMA of its own whose
//   product is added only to the cells with z <= W_r.
//   Every cell sums exactly its kept pairs.  K chunks that no cell of the
//   workgroup's tile keeps are not loaded into LDS.  With the window off the
//   kernel is compiled without any of this.
//
// Softmax: fp32 in the log2 domain.  The running max is raised only when a row's
// tile max exceeds it by more than kRescale (log2 units); otherwise the stale
// max is kept, probabilities are at most 2^kRescale, and the output and
// normaliser need no rescaling -- the result is the same softmax.  Row sums add
// the fp32 probabilities; the PV MFMA consumes them rounded to bf16.
#include "atf_internal.hpp"
#include "rope.hpp"

#include <type_traits>

namespace atf {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) char lds_char;
typedef __attribute__((address_space(3))) u32x4_t lds_u32x4;

constexpr int kBN = 64;           // keys per tile
constexpr float kRescale = 8.0f;  // lazy-rescale threshold, log2 units

// 8 waves (256 rows) per workgroup, two waves per SIMD, three LDS stages; the
// windowed kernel at d = 64 instead runs 4 waves (128 rows) per workgroup with two
// LDS stages, so that three workgroups share a CU at its ~160 VGPRs.
template <int D, bool kWin>
struct Cfg {
    static constexpr bool kSmall = D == 64 && kWin;
    static constexpr int kWaves = kSmall ? 4 : 8;
    static constexpr int kThreads = kWaves * 64;
    static constexpr int kRows = kWaves * 32;  // query rows per workgroup
    static constexpr int kStages = kSmall ? 2 : 3;  // LDS buffers per K and V tile
    static constexpr int kMinWavesPerSimd = kSmall ? 3 : 2;
    static constexpr int kHalf = D / 2;
    static constexpr int kChunks = D / 16;
    static constexpr int kKTile = kChunks * kBN * 16;  // bf16; [chunk][block][half][key][8]
    static constexpr int kVBlkBytes = D * 32;          // one packed 16-key V block [d][16]
    static constexpr int kVTile = kBN * D;             // bf16; four packed blocks
    static constexpr int kKPerWave = 2 * kChunks / kWaves;  // K (chunk, block) units per wave
    static constexpr int kVLoads = kVTile / 512;      // wave-wide 1 KB loads per V tile
    static constexpr int kVPer = (kVLoads + kWaves - 1) / kWaves;
    static_assert((2 * kChunks) % kWaves == 0, "K units must spread evenly over the waves");
    static_assert(kVTile % 512 == 0, "V tile must be whole kilobytes");
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

// LDS reads at a byte address.  Callers form addresses as (per-lane base below
// 2^18) + (constant), so the compiler folds the constants into the
// instructions' offset fields.
__device__ __forceinline__ u32x4_t lds_read_b128(uint32_t byte_addr) {
    return *(const lds_u32x4*)(uintptr_t)byte_addr;
}
// byte offset of the LDS buffer of a tile.  Passed through readfirstlane so the
// compiler treats it as one opaque scalar per tile instead of re-deriving it in
// every address (which defeats the offset-field folding above).
template <int kStages>
__device__ __forceinline__ uint32_t stage_off(int tile, int buf_bytes) {
    return uint32_t(__builtin_amdgcn_readfirstlane((tile % kStages) * buf_bytes));
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return uint32_t(reinterpret_cast<uintptr_t>((const lds_char*)p)) & 0x3FFFFu;
}

// 16 bytes per lane from global memory straight into LDS: lane i reads base + off
// (base wave-uniform) and its 16 bytes land at byte lds_wave + 16 * i (lds_wave
// wave-uniform).  Issued as inline assembly so that the compiler does not make
// LDS reads of other buffers wait for it; completion is awaited explicitly
// (vm_wait) before the workgroup barrier that publishes the buffer.
__device__ __forceinline__ void load_to_lds(const char* base, uint32_t off, uint32_t lds_wave) {
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
                 :
                 : "v"(off), "s"(base), "s"(lds_wave)
                 : "memory", "m0");
}
// wait until this wave's vector memory loads have completed (vmcnt 0 only)
__device__ __forceinline__ void vm_wait() { __builtin_amdgcn_s_waitcnt(0x0F70); }
// workgroup barrier without a memory fence: every LDS read is consumed (waited
// for) before it, and the direct-to-LDS loads are awaited with vm_wait
__device__ __forceinline__ void barrier() { __builtin_amdgcn_s_barrier(); }

// LDS of the rotation tables of the kernels that rotate at read time (dynamic, bytes)
template <int D, bool kWin>
struct RotLds {
    static constexpr int kColStride = D + 4;
    static constexpr unsigned kBytes =
        unsigned(32 * kColStride + Cfg<D, kWin>::kWaves * Cfg<D, kWin>::kKPerWave * 16 + D) * 4u;
};

// Two waves per SIMD (one workgroup per CU): the windowed kernel's registers
// exceed the 128 that four waves per SIMD would leave each wave, even at d = 64.
template <int D, bool kWin, bool kRot>
__global__ __launch_bounds__((Cfg<D, kWin>::kThreads), (Cfg<D, kWin>::kMinWavesPerSimd)) void
prefill_kernel(const std::conditional_t<kRot, PrefillRotParams, PrefillParams> p) {
    using C = Cfg<D, kWin>;
    __shared__ __attribute__((aligned(16))) uint16_t Ks[C::kStages][C::kKTile];
    __shared__ __attribute__((aligned(16))) uint16_t Vs[C::kStages][C::kVTile];
    // rotation at read time (dynamic LDS, after the static buffers): cos and sin of
    // kk * theta_r for the 32 key offsets of a 32-key block (row kk: pairs interleaved
    // as (cos, sin), padded by 16 bytes), then per wave and K unit the cos and sin of
    // the block's first position * theta_r, then rho_r (hi, lo) of every pair
    constexpr int kColStride = RotLds<D, kWin>::kColStride;
    extern __shared__ __attribute__((aligned(16))) float s_rot[];
    float* const s_colcs = s_rot;
    float* const s_base = s_rot + 32 * kColStride;
    uint2* const s_rho = reinterpret_cast<uint2*>(s_base + C::kWaves * C::kKPerWave * 16);

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

    // K: pair-chunk-major streams of cache_tokens keys, chunk c of this head =
    // 32 bytes per key; V: rows of h_kv * d bf16
    const int64_t chunk_bytes = int64_t(p.cache_tokens) * 32;
    const char* kpcm = reinterpret_cast<const char*>(p.k) + (int64_t(b) * p.h_kv + g) * C::kChunks * chunk_bytes;
    const uint32_t k_piece = uint32_t((lane & 31) * 32 + (lane >> 5) * 16);
    // V: packed 16-key blocks [d][16] of this head, ceil(cache_tokens / 16) of them
    const int n_vblk = (p.cache_tokens + 15) / 16;
    const char* vhead = reinterpret_cast<const char*>(p.v) + (int64_t(b) * p.h_kv + g) * n_vblk * int64_t(C::kVBlkBytes);

    // query fragments (B operand): row `col`, dims of half hh of every chunk
    u32x4_t qf[C::kChunks];
    {
        const uint16_t* qrow =
            p.q + ((int64_t(b) * p.n_q + my_qrow) * p.h_q + my_head) * D + hh * C::kHalf;
#pragma unroll
        for (int c = 0; c < C::kChunks; ++c) {
            u32x4_t z = {0u, 0u, 0u, 0u};
            if (row_ok) z = *reinterpret_cast<const u32x4_t*>(qrow + 8 * c);
            // an unrotated query is turned to its position here, once
            if constexpr (kRot)
                z = rope::rotate(z, rope::other_half(z, hh), hh, uint32_t(my_pos), &p.rope_rho_hi[8 * c],
                                 &p.rope_rho_lo[8 * c]);
            qf[c] = z;
        }
    }

    // ---- global -> LDS staging of the tile at key j0 into buffer `buf`.
    // K: the tile is 2 * kChunks units (chunk u / 2, 32-key block u % 2); wave w
    // loads units w, w + 8, ...: lane i reads 16 bytes of key i % 32, half i / 32,
    // so the wave's 1 KB of global memory is contiguous.  A unit whose chunk no
    // cell of the workgroup tile keeps is skipped; the last chunk is always loaded
    // because the QK of a block always multiplies it.  V: the tile's four packed
    // blocks are one contiguous run; wave w copies its kilobytes w, w + W, ...
    // Blocks past the cache's last one re-read that block (their keys are past
    // n_k and masked).
    const uint32_t ks_lds = lds_addr(&Ks[0][0]);
    const uint32_t vs_lds = lds_addr(&Vs[0][0]);
    auto tile_need = [&](int j0) __attribute__((always_inline)) -> uint32_t {
        if (!kWin) return (1u << C::kChunks) - 1u;
        const int zlo = max(0, pos_first - (j0 + kBN - 1));
        uint32_t need = 1u << (C::kChunks - 1);
#pragma unroll
        for (int c = 0; c < C::kChunks; ++c)
            if (p.win.chunk_max[c] >= zlo) need |= 1u << c;
        return need;
    };
    // Fast form for tiles wholly below n_k (all but the last): per wave unit, the
    // stream base and the first tile from which its chunk is kept (chunk c is kept in
    // the tile at j0 iff chunk_max[c] >= pos_first - j0 - 63; the thresholds are >= 0)
    // are fixed, so a tile costs one compare and one 64-bit add per load.
    const char* kbase[C::kKPerWave];
    int kfirst[C::kKPerWave];
#pragma unroll
    for (int t = 0; t < C::kKPerWave; ++t) {
        const int u = wave + C::kWaves * t;
        const int c = u >> 1;
        kbase[t] = kpcm + c * chunk_bytes + (u & 1) * 1024;
        kfirst[t] = 0;
        if (kWin && c != C::kChunks - 1) {
            const int64_t num = int64_t(pos_first) - (kBN - 1) - p.win.chunk_max[c];
            kfirst[t] = num <= 0 ? 0 : int(min(int64_t(INT32_MAX), (num + kBN - 1) / kBN));
        }
    }
    auto issue_fast = [&](int j0, int buf) __attribute__((always_inline)) -> uint32_t {
        uint32_t loaded = 0;
        const int tn = j0 / kBN;
        const int64_t koff = int64_t(j0) * 32;
        const int64_t voff = int64_t(j0) * (2 * D);
        const uint32_t kdst = ks_lds + uint32_t(buf * C::kKTile * 2);
#pragma unroll
        for (int t = 0; t < C::kKPerWave; ++t) {
            const int u = wave + C::kWaves * t;
            if (tn >= kfirst[t]) {
                load_to_lds(kbase[t] + koff, k_piece, kdst + 1024u * u);
                loaded |= 1u << t;
            }
        }
        const uint32_t vdst = vs_lds + uint32_t(buf * C::kVTile * 2);
#pragma unroll
        for (int t = 0; t < C::kVPer; ++t) {
            const int u = wave + C::kWaves * t;
            if constexpr (C::kVLoads % C::kWaves != 0)
                if (u >= C::kVLoads) break;
            load_to_lds(vhead + voff + 1024 * u, uint32_t(lane) * 16u, vdst + 1024u * u);
        }
        return loaded;
    };
    // returns the K units (bit t: unit wave + kWaves t) this wave loaded
    auto issue = [&](int j0, int buf) __attribute__((always_inline)) -> uint32_t {
        if (j0 + kBN <= p.n_k) return issue_fast(j0, buf);
        uint32_t loaded = 0;
        const uint32_t need = tile_need(j0);
        const uint32_t kdst = ks_lds + uint32_t(buf * C::kKTile * 2);
#pragma unroll
        for (int t = 0; t < C::kKPerWave; ++t) {
            const int u = wave + C::kWaves * t;  // unit = (chunk u / 2, 32-key block u % 2)
            const int c = u >> 1;
            if ((need >> c) & 1u) {
                const int jb = min(j0 + 32 * (u & 1), p.n_k - 1);
                uint32_t off = k_piece;
                if (jb + 32 > p.n_k)
                    off = min(uint32_t(lane & 31), uint32_t(p.n_k - 1 - jb)) * 32u + uint32_t(lane >> 5) * 16u;
                load_to_lds(kpcm + c * chunk_bytes + int64_t(jb) * 32, off, kdst + 1024u * u);
                loaded |= 1u << t;
            }
        }
        const uint32_t vdst = vs_lds + uint32_t(buf * C::kVTile * 2);
#pragma unroll
        for (int t = 0; t < C::kVPer; ++t) {
            const int u = wave + C::kWaves * t;
            if (u >= C::kVLoads) break;
            const int blk = min(j0 / 16 + (1024 * u) / C::kVBlkBytes, n_vblk - 1);
            load_to_lds(vhead + int64_t(blk) * C::kVBlkBytes + (1024 * u) % C::kVBlkBytes,
                        uint32_t(lane) * 16u, vdst + 1024u * u);
        }
        return loaded;
    };

    // ---- rotation at read time: each wave turns the K units it loaded, once they have
    // landed and before the barrier that publishes the tile, so each kept (key, pair) of
    // the workgroup's tile is rotated once and pruned chunks (never loaded) never are.
    // Lane l turns 4 pairs (half l / 32 of the unit's 8) of key l % 32: both components
    // from the unit's two halves, angle (block start + l % 32) * theta_r by angle
    // addition of the block start's angle (lanes 0 .. 8 kKPerWave - 1, one pair of one
    // unit each) and the offset's (the table).
    auto rotate_units = [&](int j0, int buf, uint32_t loaded) __attribute__((always_inline)) {
        loaded = __builtin_amdgcn_readfirstlane(loaded);
        if (loaded == 0u) return;
        // block-start angles of all the wave's units at once: lane 8 t + e holds pair
        // 8 c + e of unit t (c its chunk); a unit not loaded gets an unused angle
        if (lane < 8 * C::kKPerWave) {
            const int u = wave + C::kWaves * (lane >> 3);
            const float ub = rope::revolutions(uint32_t(j0 + 32 * (u & 1)), s_rho[8 * (u >> 1) + (lane & 7)]);
            s_base[wave * C::kKPerWave * 16 + 2 * lane] = __builtin_amdgcn_cosf(ub);
            s_base[wave * C::kKPerWave * 16 + 2 * lane + 1] = __builtin_amdgcn_sinf(ub);
        }
        // the wave's own LDS writes complete before its later LDS reads; the fences
        // keep the compiler from moving the reads above the writes
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        // every unit's elements are read before any is rotated, so the reads' latencies
        // overlap (reading a unit that was not loaded is harmless: it is not written)
        typedef __attribute__((address_space(3))) uint64_t lds_u64;
        const int kk = lane & 31, gq = lane >> 5;
        uint64_t xv[C::kKPerWave], yv[C::kKPerWave];
#pragma unroll
        for (int t = 0; t < C::kKPerWave; ++t) {
            const int u = wave + C::kWaves * t;
            const uint32_t a0 = ks_lds + uint32_t(buf * C::kKTile * 2) + 1024u * u + uint32_t(kk * 16 + gq * 8);
            xv[t] = *(const lds_u64*)(uintptr_t)a0;
            yv[t] = *(const lds_u64*)(uintptr_t)(a0 + 512u);
        }
#pragma unroll
        for (int t = 0; t < C::kKPerWave; ++t) {
            if (!((loaded >> t) & 1u)) continue;
            const int u = wave + C::kWaves * t;
            const float* cr = &s_colcs[kk * kColStride + 2 * (8 * (u >> 1) + 4 * gq)];
            const float4 cc0 = *reinterpret_cast<const float4*>(cr);
            const float4 cc1 = *reinterpret_cast<const float4*>(cr + 4);
            const float* br = &s_base[(wave * C::kKPerWave + t) * 16 + 8 * gq];
            const float4 bb0 = *reinterpret_cast<const float4*>(br);
            const float4 bb1 = *reinterpret_cast<const float4*>(br + 4);
            const float cC[4] = {cc0.x, cc0.z, cc1.x, cc1.z}, sC[4] = {cc0.y, cc0.w, cc1.y, cc1.w};
            const float cB[4] = {bb0.x, bb0.z, bb1.x, bb1.z}, sB[4] = {bb0.y, bb0.w, bb1.y, bb1.w};
            uint32_t xo[2], yo[2];
#pragma unroll
            for (int w2 = 0; w2 < 2; ++w2) {
                const uint32_t xw = uint32_t(xv[t] >> (32 * w2)), yw = uint32_t(yv[t] >> (32 * w2));
                rope::bf16x2_t xt, yt;
#pragma unroll
                for (int h = 0; h < 2; ++h) {
                    const int e = 2 * w2 + h;
                    const float cs = __builtin_fmaf(cB[e], cC[e], -sB[e] * sC[e]);
                    const float sn = __builtin_fmaf(sB[e], cC[e], cB[e] * sC[e]);
                    const float x = __uint_as_float(h ? (xw & 0xFFFF0000u) : (xw << 16));
                    const float y = __uint_as_float(h ? (yw & 0xFFFF0000u) : (yw << 16));
                    xt[h] = (__bf16)rope::turn(x, y, -1.f, cs, sn);
                    yt[h] = (__bf16)rope::turn(y, x, 1.f, cs, sn);
                }
                xo[w2] = __builtin_bit_cast(uint32_t, xt);
                yo[w2] = __builtin_bit_cast(uint32_t, yt);
            }
            const uint32_t a0 = ks_lds + uint32_t(buf * C::kKTile * 2) + 1024u * u + uint32_t(kk * 16 + gq * 8);
            *(lds_u64*)(uintptr_t)a0 = uint64_t(xo[0]) | (uint64_t(xo[1]) << 32);
            *(lds_u64*)(uintptr_t)(a0 + 512u) = uint64_t(yo[0]) | (uint64_t(yo[1]) << 32);
        }
        // the rotated units are complete in LDS before the workgroup barrier, and the
        // fence keeps the compiler from sinking the writes below it
        __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    };
    // after the barrier: no LDS read of a rotated unit moves above it
    auto rotated_acquire = [&]() __attribute__((always_inline)) {
        if constexpr (kRot) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    };

    // per-lane LDS byte bases of the fragment reads (buffer 0, block 0)
    //   K: unit (chunk c, block kb) at 1 KB * (2 c + kb), half hh, key col
    //   V: packed block q of the tile at q * kVBlkBytes, dim 32 i + col at 1 KB * i,
    //      slots 8 hh .. 8 hh + 7
    const uint32_t k_lane = ks_lds + uint32_t(hh * 512 + col * 16);
    const uint32_t v_lane = vs_lds + uint32_t(col * 32 + hh * 16);

    f32x16_t oacc[D / 32];
#pragma unroll
    for (int i = 0; i < D / 32; ++i) oacc[i] = zero16();
    float m_run = -INFINITY;  // running (possibly stale) max, log2 domain
    float m_thr = -INFINITY;  // m_run + kRescale: a tile max above it raises m_run
    float m_neg = 0.f;        // minus the max the exponentials subtract (0 while m_run = -inf)
    float l_run = 0.f;        // normaliser over this lane's keys
    const float sc = p.scale_log2;
    f32x16_t sacc[2];  // scores of the current tile (two 32-key blocks)
    u32x4_t qb;        // query dims of chunk qb_rf / 8 with the pairs below qb_rf zeroed
    int qb_rf = -1;

    auto k_block = [&](int tile, int kb) __attribute__((always_inline)) -> uint32_t {
        return k_lane + stage_off<C::kStages>(tile, C::kKTile * 2) + uint32_t(kb * 1024);
    };

    // ---- QK of a uniform tile: chunk CF with the boundary operand qb, then the
    // whole chunks above it (for the window off: CF = 0, qb = qf[0])
    auto qk_uniform = [&](int tile, auto cf_tag) __attribute__((always_inline)) {
        constexpr int CF = decltype(cf_tag)::value;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const uint32_t kr = k_block(tile, kb);
            u32x4_t kf[C::kChunks];
#pragma unroll
            for (int c = CF; c < C::kChunks; ++c) kf[c] = lds_read_b128(kr + 2048u * c);
            f32x16_t acc = mfma(kf[CF], qb, zero16());
#pragma unroll
            for (int c = CF + 1; c < C::kChunks; ++c) acc = mfma(kf[c], qf[c], acc);
            sacc[kb] = acc;
        }
    };

    // ---- QK of any tile (general path), per 32-key block
    auto qk_general = [&](int tile) __attribute__((always_inline)) {
        const int j0 = tile * kBN;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            const int jb = j0 + 32 * kb;
            const uint32_t kr = k_block(tile, kb);
            u32x4_t kf[C::kChunks];
#pragma unroll
            for (int c = 0; c < C::kChunks; ++c) kf[c] = lds_read_b128(kr + 2048u * c);
            const int zhi = wp_max - jb;
            const int zlo = max(0, wp_min - (jb + 31));
            // all pairs classified at once: lane r holds W_r; bit r of `full` = pair r
            // kept in every cell of the block, of `keep` = kept in some cell
            const uint64_t full = __ballot(my_w >= zhi);
            const uint64_t keep = __ballot(my_w >= zlo);
            // lowest frequencies (largest windows) first: the first MFMA always runs
            // (pairs no cell keeps zeroed) and starts from a zero accumulator
            f32x16_t acc;
#pragma unroll
            for (int c = C::kChunks - 1; c >= 0; --c) {
                const uint32_t fc = uint32_t(full >> (8 * c)) & 0xFFu;
                if (c == C::kChunks - 1) {
                    acc = mfma(kf[c], keep_pairs(qf[c], fc), zero16());
                } else if (fc) {
                    u32x4_t q = qf[c];
                    if (fc != 0xFFu) q = keep_pairs(q, fc);
                    acc = mfma(kf[c], q, acc);
                }
            }
            // pairs whose window ends inside the block, grouped by chunk and threshold:
            // one MFMA per group, added where z <= W_r (register v holds distance
            // zbase - off(v): keep iff off(v) >= thr).  A table whose chunks share one
            // threshold (the rounded slice) needs one MFMA per partial chunk.
            uint64_t part = keep & ~full;
            while (part) {
                const int r = __builtin_ctzll(part);
                const int c = r >> 3;
                const int wr = p.win.W[r];
                const uint64_t grp = __ballot(my_w == wr) & part & (0xFFull << (8 * c));
                part &= ~grp;
                u32x4_t qc = qf[0];
#pragma unroll
                for (int cc = 1; cc < C::kChunks; ++cc)
                    if (cc == c) qc = qf[cc];
                const f32x16_t pr = mfma(lds_read_b128(kr + 2048u * c),
                                         keep_pairs(qc, uint32_t(grp >> (8 * c))), zero16());
                const int thr = my_pos - jb - 4 * hh - wr;
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int off = 8 * (v / 4) + (v % 4);
                    acc[v] += off >= thr ? pr[v] : 0.f;
                }
            }
            sacc[kb] = acc;
        }
    };

    // ---- causal mask and key bound (only tiles that reach the diagonal or n_k),
    // then the online softmax over the tile (lane = query row; the two lane halves
    // hold disjoint keys), then PV.  One rescale check per tile; the exponentials
    // are branch-free.
    auto softmax_pv = [&](int tile) __attribute__((always_inline)) {
        const int j0 = tile * kBN;
        if (wp_min - (j0 + kBN - 1) < 0 || j0 + kBN > p.n_k) {
            // cell kept iff off <= lim = min(distance base, last key - block start): the
            // score goes through min(s, +inf) if kept, min(s, -inf) if not, the sign bit of
            // lim - off choosing the infinity.  (Written with per-cell compares, the 32
            // lane masks of a tile were all live at once and pushed the kernel's scalar
            // registers into spills.)
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                const int jb = j0 + 32 * kb;
                const int lim = min(my_pos - jb, p.n_k - 1 - jb) - 4 * hh;
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int off = 8 * (v / 4) + (v % 4);
                    const uint32_t inf = (uint32_t(lim - off) & 0x80000000u) | 0x7F800000u;
                    sacc[kb][v] = fminf(sacc[kb][v], __uint_as_float(inf));
                }
            }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[kb][v]);
        // The two lane halves of a row hold the same m_run and sc > 0, so some lane's half
        // max passes the threshold exactly when some lane's row max does: the halves
        // exchange their maxima only when the running max is raised.
        if (__any(mx * sc > m_thr)) {
            mx = fmaxf(mx, __shfl_xor(mx, 32));
            const float m_new = fmaxf(m_run, mx * sc);
            const float m_use = m_new == -INFINITY ? 0.f : m_new;
            const float alpha = exp2_fast(m_run - m_use);
            m_run = m_new;
            m_thr = m_new + kRescale;
            m_neg = -m_use;
            l_run *= alpha;
#pragma unroll
            for (int i = 0; i < D / 32; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v) oacc[i][v] *= alpha;
        }
        const uint32_t vb = v_lane + stage_off<C::kStages>(tile, C::kVTile * 2);
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
            u32x4_t pb[2];
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                for (int t = 0; t < 4; ++t) {
                    const float a = exp2_fast(__builtin_fmaf(sacc[kb][8 * ks + 2 * t], sc, m_neg));
                    const float c2 = exp2_fast(__builtin_fmaf(sacc[kb][8 * ks + 2 * t + 1], sc, m_neg));
                    l_run += a;
                    l_run += c2;
                    bf16x2_t two;
                    two[0] = (__bf16)a;
                    two[1] = (__bf16)c2;
                    pb[ks][t] = __builtin_bit_cast(uint32_t, two);
                }
#pragma unroll
            for (int ks = 0; ks < 2; ++ks)
#pragma unroll
                for (int i = 0; i < D / 32; ++i)
                    oacc[i] = mfma(lds_read_b128(vb + uint32_t((2 * kb + ks) * C::kVBlkBytes + 1024 * i)),
                                   pb[ks], oacc[i]);
        }
    };

    // The V slots of keys at or past n_k in the LDS copy of a tile that crosses n_k
    // (only the last tile can) are set to zero by the whole workgroup before any
    // wave reads them: the cache past n_k need not hold finite values, and a zero
    // probability does not cancel a NaN in the matrix product.
    auto zero_v_tail = [&](int u) __attribute__((always_inline)) {
        const int j0 = u * kBN;
        if (j0 + kBN <= p.n_k) return;
        uint16_t* vt = &Vs[u % C::kStages][0];
        for (int row = tid; row < 4 * D; row += C::kThreads) {  // row = block * D + dim
            const int kblk = j0 + 16 * (row / D);
#pragma unroll
            for (int sl = 0; sl < 16; ++sl) {
                const int key = kblk + 8 * ((sl & 7) >> 2) + 4 * (sl >> 3) + (sl & 3);
                if (key >= p.n_k) vt[row * 16 + sl] = 0;
            }
        }
        __syncthreads();
    };

    const int n_tiles = (key_end + kBN - 1) / kBN;
    auto active = [&](int tile) __attribute__((always_inline)) { return wave_active && wp_max >= tile * kBN; };
    // one tile: stage the next, compute this one (if the wave has rows there),
    // await this wave's loads of the next tile (and rotate them, for unrotated
    // caches), barrier
    auto run_tile = [&](int u, auto&& qk) __attribute__((always_inline)) {
        uint32_t loaded = 0;
        if (u + 1 < n_tiles) loaded = issue((u + 1) * kBN, (u + 1) % C::kStages);
        zero_v_tail(u);
        if (active(u)) {
            qk(u);
            softmax_pv(u);
        }
        vm_wait();
        if constexpr (kRot) rotate_units((u + 1) * kBN, (u + 1) % C::kStages, loaded);
        barrier();
        rotated_acquire();
    };

    if constexpr (kRot) {
        for (int idx = tid; idx < 32 * C::kHalf; idx += C::kThreads) {
            const int kk = idx / C::kHalf, r = idx % C::kHalf;
            const float u = rope::revolutions(uint32_t(kk), make_uint2(p.rope_rho_hi[r], p.rope_rho_lo[r]));
            s_colcs[kk * kColStride + 2 * r] = __builtin_amdgcn_cosf(u);
            s_colcs[kk * kColStride + 2 * r + 1] = __builtin_amdgcn_sinf(u);
        }
        if (tid < C::kHalf) s_rho[tid] = make_uint2(p.rope_rho_hi[tid], p.rope_rho_lo[tid]);
        __syncthreads();
    }
    {
        const uint32_t loaded = issue(0, 0);
        vm_wait();
        if constexpr (kRot) rotate_units(0, 0, loaded);
        barrier();
        rotated_acquire();
    }

    if constexpr (!kWin) {
        // window off: every tile is the full contraction
        qb = qf[0];
        for (int u = 0; u < n_tiles; ++u)
            run_tile(u, [&](int t) __attribute__((always_inline)) {
                qk_uniform(t, std::integral_constant<int, 0>{});
            });
    } else {
    // Each wave walks the tiles in runs; every tile ends with one barrier on every
    // wave, whichever loop runs it.
    constexpr int kGeneral = 64;  // mode of a general-path tile (chunk counts are 0..7)
    int u = 0;
    while (u < n_tiles) {
        int mode, seg_end;
        if (!active(u)) {
            mode = -1;  // the wave's rows all precede this tile and every later one
            seg_end = n_tiles;
        } else {
            mode = kGeneral;
            seg_end = u + 1;
            if (p.mono) {
                const int zhi = wp_max - u * kBN;                      // largest distance of the tile
                const int zlo = max(0, wp_min - (u * kBN + kBN - 1));  // smallest
                const uint64_t full = __ballot(my_w >= zhi);
                const uint64_t keep = __ballot(my_w >= zlo);
                if (full == keep) {
                    // uniform: kept pairs r >= rf (non-empty: the last chunk is kept at
                    // every distance of the call).  The run lasts while the next
                    // threshold below, W[rf - 1], stays under the tile's smallest
                    // distance: wp_min - 64 u' - 63 > W[rf - 1].
                    const int rf = __builtin_ctzll(full);
                    seg_end = n_tiles;
                    if (rf > 0) {
                        const int wlow = p.win.W[rf - 1];
                        const int64_t lim = (int64_t(wp_min) - kBN - wlow) / kBN + 1;
                        seg_end = int(max(int64_t(u) + 1, min(lim, int64_t(n_tiles))));
                    }
                    mode = rf >> 3;
                    if (rf != qb_rf) {
                        qb_rf = rf;
                        u32x4_t qs = qf[0];
#pragma unroll
                        for (int cc = 1; cc < C::kChunks; ++cc)
                            if (cc == (rf >> 3)) qs = qf[cc];
                        qb = keep_pairs(qs, (0xFFu << (rf & 7)) & 0xFFu);
                    }
                }
            }
        }
        switch (mode) {
#define ATF_UNIFORM_RUN(CFV)                                                                    \
    case CFV:                                                                                   \
        if constexpr (CFV < C::kChunks) {                                                       \
            for (; u < seg_end; ++u)                                                            \
                run_tile(u, [&](int t) __attribute__((always_inline)) { qk_uniform(t, std::integral_constant<int, CFV>{}); }); \
        } else { /* not reached: rf < d/2 - 8 */                                                \
            run_tile(u, [&](int t) __attribute__((always_inline)) { qk_general(t); });                                         \
            ++u;                                                                                \
        }                                                                                       \
        break;
            ATF_UNIFORM_RUN(0)
            ATF_UNIFORM_RUN(1)
            ATF_UNIFORM_RUN(2)
            ATF_UNIFORM_RUN(3)
            ATF_UNIFORM_RUN(4)
            ATF_UNIFORM_RUN(5)
            ATF_UNIFORM_RUN(6)
            ATF_UNIFORM_RUN(7)
#undef ATF_UNIFORM_RUN
            case kGeneral:
                run_tile(u, [&](int t) __attribute__((always_inline)) { qk_general(t); });
                ++u;
                break;
            default:  // idle: keep the barrier count
                for (; u < seg_end; ++u) {
                    uint32_t loaded = 0;
                    if (u + 1 < n_tiles) loaded = issue((u + 1) * kBN, (u + 1) % C::kStages);
                    zero_v_tail(u);
                    vm_wait();
                    if constexpr (kRot) rotate_units((u + 1) * kBN, (u + 1) % C::kStages, loaded);
                    barrier();
                    rotated_acquire();
                }
                break;
        }
    }
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

template <int D, bool kRot, class P>
hipError_t launch_d(const P& p, unsigned blocks, bool window_on, hipStream_t stream) {
    constexpr unsigned kLdsOn = kRot ? RotLds<D, true>::kBytes : 0u;
    constexpr unsigned kLdsOff = kRot ? RotLds<D, false>::kBytes : 0u;
    if (window_on)
        hipLaunchKernelGGL((prefill_kernel<D, true, kRot>), dim3(blocks), dim3(Cfg<D, true>::kThreads),
                           kLdsOn, stream, p);
    else
        hipLaunchKernelGGL((prefill_kernel<D, false, kRot>), dim3(blocks),
                           dim3(Cfg<D, false>::kThreads), kLdsOff, stream, p);
    return hipGetLastError();
}

// Tile geometry and the uniform-run test, shared by both launchers.
template <class P>
hipError_t prepare(P& p, int head_dim, unsigned* blocks, bool* window_on) {
    // the window is off when no threshold is below the largest possible distance;
    // the uniform-run path needs thresholds non-decreasing in r and the last chunk
    // kept at every distance of the call
    const int64_t max_dist = int64_t(p.q_pos0) + p.n_q - 1;
    bool on = false;
    for (int r = 0; r < head_dim / 2; ++r)
        if (int64_t(p.win.W[r]) < max_dist) on = true;
    bool mono = int64_t(p.win.W[head_dim / 2 - kChunkPairs]) >= max_dist;
    for (int r = 1; r < head_dim / 2; ++r)
        if (p.win.W[r] < p.win.W[r - 1]) mono = false;
    p.mono = mono ? 1 : 0;
    const int rows = head_dim == 64 ? (on ? Cfg<64, true>::kRows : Cfg<64, false>::kRows)
                                    : (on ? Cfg<128, true>::kRows : Cfg<128, false>::kRows);
    if (p.group < 1 || p.group > rows) return hipErrorInvalidValue;
    p.pos_per_tile = rows / p.group;
    p.n_qtiles = (p.n_q + p.pos_per_tile - 1) / p.pos_per_tile;
    const int64_t n = int64_t(p.n_qtiles) * p.h_kv * p.batch;
    if (n <= 0 || n > 0x7fffffff) return hipErrorInvalidConfiguration;
    *blocks = unsigned(n);
    *window_on = on;
    (void)hipGetLastError();
    return hipSuccess;
}

}  // namespace

hipError_t launch_prefill(const PrefillParams& p_in, int head_dim, hipStream_t stream) {
    PrefillParams p = p_in;
    unsigned blocks = 0;
    bool window_on = false;
    const hipError_t e = prepare(p, head_dim, &blocks, &window_on);
    if (e != hipSuccess) return e;
    return head_dim == 64 ? launch_d<64, false>(p, blocks, window_on, stream)
                          : launch_d<128, false>(p, blocks, window_on, stream);
}

hipError_t launch_prefill_rotating(const PrefillRotParams& p_in, int head_dim, hipStream_t stream) {
    PrefillRotParams p = p_in;
    unsigned blocks = 0;
    bool window_on = false;
    const hipError_t e = prepare(p, head_dim, &blocks, &window_on);
    if (e != hipSuccess) return e;
    return head_dim == 64 ? launch_d<64, true>(p, blocks, window_on, stream)
                          : launch_d<128, true>(p, blocks, window_on, stream);
}

}  // namespace atf
