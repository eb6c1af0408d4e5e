// Windowed single-token decode for gfx950: split-KV with partial online-softmax
// states and a merge kernel (the decode form of Fig. fa is the last query row;
// the split/merge decomposition is the one Sec. 5 describes), over a
// pair-chunk-major K cache so that pruned pairs are never read from HBM.
//
// Caches (both produced from [B][n_k][h_kv][d] by the pack kernels below):
//   K [B][h_kv][d/16][n_k][16]: chunk c of a head is a contiguous stream over
//     tokens of 16 bf16 = dims [8c, 8c+8) then [d/2 + 8c, d/2 + 8c + 8).  With the
//     query at position q_pos, token t sits at distance z = q_pos - t, and chunk c
//     is needed only where z <= max_{r in c} W_r: a contiguous suffix of its
//     stream.  32 tokens of one chunk are 1 KB of contiguous memory.
//   V [B][h_kv][ceil(n_k/16)][d][16]: blocks of 16 tokens stored d-major, the 16
//     tokens of a d-row in the order the PV matrix instruction consumes them
//     (position 8h + e holds token 8*(e/4) + 4h + e%4), zero past n_k.
//
// The G query heads of one KV head are the columns of 32x32 MFMA tiles, so a
// decode step is the prefill's arithmetic with "query rows" = heads:
//   S^T[token][head] = K[token][dims] * Q^T[dims][head]   (A from the K stream)
//   O^T[d][head]    += V^T[d][token] * P^T[token][head]   (A from the V blocks)
// Every operand fragment is a 16-byte load straight from HBM into registers; no
// LDS staging and no barrier in the streaming loop.  Each wave streams its own
// 32-token blocks of the workgroup's split; the four waves' partial softmax
// states are combined in LDS and written as the split's partial.
//
// Window: per 32-token block, all pairs are classified by two lane-parallel
// compares and ballots (lane r holds W_r): pairs kept at every distance of the
// block, and pairs kept at some distance.  Chunks with no kept pair are not
// loaded.  Pairs whose window ends inside the block get one extra MFMA each,
// added only to the tokens within their window.
//
// Batches: a uniform batch splits every row into the same token ranges; a ragged or
// paged batch (row lengths in device arrays) cuts the batch's keys into equal spans,
// each row into whole spans of its own keys, laid out by every workgroup from the row
// arrays (ragged_item).
//
// Rotation at read time (App. B): with unrotated q and K the kernel applies RoPE to
// the query once and to each key chunk it loads, so a pruned pair is neither read nor
// rotated.
#include "atf_internal.hpp"
#include "rope.hpp"

#include <mutex>

namespace atf {
namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int kWaves = 4;
constexpr float kRescale = 8.0f;  // lazy-rescale threshold, log2 units

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

// Keep only the pairs whose bit is set in `mask` (bit e = pair 8c+e of the chunk).
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

// Keys of ragged row r that its query reaches (the clamps keep every read inside the
// row's cache): min(n_k_rows[r], q_pos_rows[r] + 1), within [0, n_k].
__device__ __forceinline__ int ragged_valid(const DecodeParams& p, int r) {
    const int nk = min(max(p.n_k_rows[r], 0), p.n_k);
    const int qp = min(max(p.q_pos_rows[r], 0), 0x7FFFFFFD);
    return min(nk, qp + 1);
}

// Work plan of a ragged batch, the same in every wave that computes it: the batch's
// causal keys are cut into spans of `span` tokens (about total / p.splits, a multiple
// of the workgroup's token step), each row into ceil(n_valid / span) items of its own
// keys, items numbered row by row.  Returns the row of `item` (or -1 past the last
// item) and its first token; with `plan` set, also writes the index of each row's
// first item and the item count at plan[B].
__device__ int ragged_item(const DecodeParams& p, int item, int& t_first, int64_t& span,
                           int32_t* plan) {
    const int lane = threadIdx.x & 63;
    int64_t total = 0;
    for (int r0 = 0; r0 < p.batch; r0 += 64) {
        int64_t nv = r0 + lane < p.batch ? ragged_valid(p, r0 + lane) : 0;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) nv += __shfl_xor(nv, o);
        total += nv;
    }
    span = (total + p.splits - 1) / p.splits;
    span = (span + kDecodeTokenStep - 1) / kDecodeTokenStep * kDecodeTokenStep;
    if (span < kDecodeTokenStep) span = kDecodeTokenStep;
    int row = -1, first = 0;
    int before = 0;  // items of the rows below r0
    for (int r0 = 0; r0 < p.batch; r0 += 64) {
        const int r = r0 + lane;
        const int cnt = r < p.batch ? int((ragged_valid(p, r) + span - 1) / span) : 0;
        int incl = cnt;  // inclusive prefix over the wave's rows
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int y = __shfl_up(incl, o);
            if (lane >= o) incl += y;
        }
        incl += before;
        if (plan != nullptr && r < p.batch) plan[r] = incl - cnt;
        const uint64_t hit = __ballot(item < incl);
        if (row < 0 && hit != 0) {
            const int l = __builtin_ctzll(hit);
            row = r0 + l;
            first = item - __shfl(incl - cnt, l);
        }
        before = __shfl(incl, 63);
    }
    if (plan != nullptr && lane == 0) plan[p.batch] = before;
    t_first = int(int64_t(first) * span);
    return row;
}

template <int D, bool kRot>
__global__ __launch_bounds__(kWaves * 64, 2) void decode_split_kernel(const DecodeParams p) {
    constexpr int kChunks = D / 16;
    constexpr int kHalf = D / 2;
    constexpr int kDB = D / 32;  // 32-dim blocks of the output
    __shared__ float red_m[kWaves][32];
    __shared__ float red_l[kWaves][32];
    __shared__ float red_o[kDecodeMaxHeads][D + 1];
    // rotation at read time: cos and sin of col * theta_r for the 32 token columns of a
    // block (row col: pairs interleaved as (cos, sin)); a key's angle is the block's
    // t0 * theta_r plus this, combined by angle addition.  Rows padded by 16 bytes so the
    // 32 columns' reads fall in different banks.
    constexpr int kCStride = 2 * kHalf + 4;
    __shared__ __attribute__((aligned(16))) float s_colcs[kRot ? 32 * kCStride : 1];
    // per wave: (cos, sin) of the current block's t0 * theta_r for every pair r, written by
    // lane r and read back by all lanes (broadcast reads of the chunk's 8 pairs)
    __shared__ __attribute__((aligned(16))) float s_blkcs[kRot ? kWaves * 2 * kHalf : 1];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int col = lane & 31;  // head column
    const int hh = lane >> 5;
    const int split = blockIdx.x;
    const int NH = p.heads_per_block;
    const int subgroups = p.group / NH;
    const int g = blockIdx.y / subgroups;
    const int sub = blockIdx.y % subgroups;
    const int hq0 = g * p.group + sub * NH;
    const bool head_ok = col < NH;

    // this workgroup's row and tokens: a uniform batch has row blockIdx.z and split
    // `split` of p.split_tokens tokens; a ragged batch gives each row its own keys and
    // query position, and blockIdx.x is a work item of the plan (ragged_item)
    int b, n_k = p.n_k, q_pos = p.q_pos, n_valid = p.n_valid, t_begin, t_end;
    int64_t slot0;  // partial-state slot of head hq0 (heads follow at stride 1)
    if (p.n_k_rows != nullptr) {
        int64_t span;
        int32_t* plan = (blockIdx.x == 0 && blockIdx.y == 0 && wave == 0) ? p.ws_plan : nullptr;
        b = ragged_item(p, split, t_begin, span, plan);
        if (b < 0) return;  // past the last item (the whole workgroup: wave-uniform)
        n_k = min(max(p.n_k_rows[b], 0), p.n_k);
        q_pos = min(max(p.q_pos_rows[b], 0), 0x7FFFFFFD);
        n_valid = min(n_k, q_pos + 1);
        t_end = int(min(int64_t(n_valid), int64_t(t_begin) + span));
        slot0 = int64_t(split) * p.h_q + hq0;
    } else {
        b = blockIdx.z;
        t_begin = split * p.split_tokens;
        t_end = min(n_valid, t_begin + p.split_tokens);
        slot0 = (int64_t(b) * p.h_q + hq0) * p.splits + split;
    }
    // the split's bounds are the same for every lane; saying so keeps the block loop's
    // exit, and the window ballots carried from one block to the next, in scalar
    // registers, so that each MFMA below is skipped by a scalar branch (an MFMA issued
    // under an all-zero EXEC mask still accumulates)
    t_begin = __builtin_amdgcn_readfirstlane(t_begin);
    t_end = __builtin_amdgcn_readfirstlane(t_end);
    const int64_t cap = p.cache_tokens;  // stream length of the caches
    const uint16_t* kstream = p.kpcm + (int64_t(b) * p.h_kv + g) * kChunks * cap * 16;
    const uint16_t* vblocks = p.vpk + (int64_t(b) * p.h_kv + g) * ((cap + 15) / 16) * D * 16;
    const int my_w = lane < kHalf ? p.win.W[lane] : -1;
    if constexpr (kRot) {
        for (int e = tid; e < 32 * kHalf; e += kWaves * 64) {
            const int cc = e / kHalf, r = e % kHalf;
            const float u = rope::revolutions(uint32_t(cc), make_uint2(p.rope_rho_hi[r], p.rope_rho_lo[r]));
            s_colcs[cc * kCStride + 2 * r] = __builtin_amdgcn_cosf(u);
            s_colcs[cc * kCStride + 2 * r + 1] = __builtin_amdgcn_sinf(u);
        }
        __syncthreads();
    }
    // lane r's pair (r < d/2): its rotation fraction, for the per-block angles
    const uint2 my_rho = kRot && lane < kHalf ? make_uint2(p.rope_rho_hi[lane], p.rope_rho_lo[lane])
                                              : make_uint2(0u, 0u);

    // query fragments (B operand): head column `col`, dims of half hh of every chunk
    // (rotated to the query position here when the query is given unrotated)
    u32x4_t qf[kChunks];
    {
        const uint16_t* qvec = p.q + (int64_t(b) * p.h_q + hq0 + (head_ok ? col : 0)) * D;
#pragma unroll
        for (int c = 0; c < kChunks; ++c) {
            u32x4_t z = {0u, 0u, 0u, 0u};
            if (head_ok) z = *reinterpret_cast<const u32x4_t*>(qvec + hh * kHalf + 8 * c);
            // (both lanes of a pair hold the same column, and zeros rotate to zeros)
            if constexpr (kRot)
                z = rope::rotate(z, rope::other_half(z, hh), hh, uint32_t(q_pos), &p.rope_rho_hi[8 * c],
                                &p.rope_rho_lo[8 * c]);
            qf[c] = z;
        }
    }

    f32x16_t oacc[kDB];
#pragma unroll
    for (int i = 0; i < kDB; ++i) oacc[i] = zero16();
    float m_run = -INFINITY;
    float m_thr = -INFINITY;  // m_run + kRescale: a block max above it raises m_run
    float m_neg = 0.f;        // minus the max the exponentials subtract (0 while m_run = -inf)
    float l_run = 0.f;
    const float sc = p.scale_log2;

    // a block's place in the caches (the row's contiguous cache, or the page the block
    // table names; a page holds a whole number of 32-token blocks) and its window
    // classification: `full` = pairs kept at every token of the block, `keep` = pairs
    // kept at one or more
    struct Blk {
        const uint16_t* kb;  // chunk c of token t at kb + (c * kstride + t - tb) * 16
        const uint16_t* vb;  // 16-token block j at vb + (j - tb / 16) * D * 16
        int64_t kstride;
        int tb;
        uint64_t full, keep;
    };
    auto locate = [&](int t0) {
        Blk B = {kstream, vblocks, cap, 0, 0ull, 0ull};
        if (p.block_table != nullptr) {
            const int pt = p.page_tokens;
            const int page = min(max(p.block_table[int64_t(b) * p.max_pages + t0 / pt], 0),
                                 p.num_pages - 1);
            B.kb = p.kpcm + (int64_t(page) * p.h_kv + g) * kChunks * int64_t(pt) * 16;
            B.vb = p.vpk + (int64_t(page) * p.h_kv + g) * (pt / 16) * int64_t(D) * 16;
            B.kstride = pt;
            B.tb = t0 - t0 % pt;
        }
        const int t_last = min(t0 + 31, t_end - 1);
        B.full = __ballot(my_w >= q_pos - t0);
        B.keep = __ballot(my_w >= max(0, q_pos - t_last));
        return B;
    };
    // K fragments of the kept chunks (A operand: token t0 + col, dims of half hh); the
    // last chunk is always fetched because the first MFMA multiplies it.
    //
    // With rotation at read time the next block's K is loaded while the current block is
    // rotated, multiplied and accumulated (its registers are free once the block's QK
    // products are issued), and the current block's V is loaded before its K is rotated.
    // The waits then have to count the loads in flight, so that count must not depend on
    // the window: a chunk no token of the block keeps re-reads the always-fetched last
    // chunk (a cache hit; its fragment is never multiplied), and a token past the split's
    // end reads the split's last token (its score is masked).  Without rotation the
    // loads are few enough in time to be issued with the block's own V, and pruned
    // chunks are not loaded at all.
    u32x4_t kf[kChunks];
    auto load_k = [&](const Blk& B, int t0) {
        if constexpr (kRot) {
            const int tok = min(t0 + col, t_end - 1);
            const uint16_t* base = B.kb + (int64_t(tok) - B.tb) * 16 + 8 * hh;
#pragma unroll
            for (int c = 0; c < kChunks; ++c) {
                const bool kept = c == kChunks - 1 || ((B.keep >> (8 * c)) & 0xFFull) != 0;
                kf[c] = *reinterpret_cast<const u32x4_t*>(base + int64_t(kept ? c : kChunks - 1) * B.kstride * 16);
            }
        } else {
            const int tok = t0 + col;
            const bool tok_ok = tok < t_end;
#pragma unroll
            for (int c = 0; c < kChunks; ++c) {
                u32x4_t z = {0u, 0u, 0u, 0u};
                const bool kept = c == kChunks - 1 || ((B.keep >> (8 * c)) & 0xFFull) != 0;
                if (kept && tok_ok)
                    z = *reinterpret_cast<const u32x4_t*>(B.kb + (int64_t(c) * B.kstride + tok - B.tb) * 16 + 8 * hh);
                kf[c] = z;
            }
        }
    };

    int t0 = t_begin + 32 * wave;
    Blk B = {kstream, vblocks, cap, 0, 0ull, 0ull};
    if constexpr (kRot) {
        if (t0 < t_end) {
            B = locate(t0);
            load_k(B, t0);
        }
    }
    for (; t0 < t_end; t0 += 32 * kWaves) {
        if constexpr (!kRot) {
            B = locate(t0);
            load_k(B, t0);
        }
        const uint64_t full = B.full;
        const uint64_t keep = B.keep;
        const uint16_t* vb = B.vb;
        const int tb = B.tb;

        // V^T fragments (A operand: dim 32 i + col, 8 tokens of half hh of each
        // 16-token group).  A block past n_k re-reads the last block holding keys and is
        // zeroed (so that both blocks always issue their loads); in the block holding
        // token n_k the slots of later tokens are zeroed (the cache past n_k need not
        // hold finite values, and their probabilities are 0).
        u32x4_t vf[2][kDB];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            const int blk = t0 / 16 + ks;
            const int blk_rd = min(blk, (n_k - 1) / 16);
#pragma unroll
            for (int i = 0; i < kDB; ++i)
                vf[ks][i] = *reinterpret_cast<const u32x4_t*>(vb + (int64_t(blk_rd - tb / 16) * D + 32 * i + col) * 16 + 8 * hh);
            if (16 * blk >= n_k) {
#pragma unroll
                for (int i = 0; i < kDB; ++i) vf[ks][i] = u32x4_t{0u, 0u, 0u, 0u};
            }
            if (16 * blk < n_k && 16 * blk + 16 > n_k) {
                const int lim = n_k - 16 * blk - 4 * hh;  // slot e valid iff 8(e/4) + e%4 < lim
#pragma unroll
                for (int i = 0; i < kDB; ++i)
#pragma unroll
                    for (int t = 0; t < 4; ++t) {
                        const int e0 = 2 * t, e1 = 2 * t + 1;
                        const uint32_t m = (8 * (e0 / 4) + e0 % 4 < lim ? 0x0000FFFFu : 0u) |
                                           (8 * (e1 / 4) + e1 % 4 < lim ? 0xFFFF0000u : 0u);
                        vf[ks][i][t] &= m;
                    }
            }
        }

        if constexpr (kRot) {
            // the keys at their positions t0 + col, rotated here: only the kept chunks
            // are read, so only their pairs are rotated (both lanes of a pair hold the
            // same token).  Angle of (t0 + col, r) by angle addition: lane r evaluates
            // the block's t0 * theta_r once and leaves its cosine and sine in the wave's
            // LDS row; every lane reads those of its chunk's 8 pairs and col * theta_r from LDS.
            const float ub = rope::revolutions(uint32_t(t0), my_rho);
            float* blk = &s_blkcs[wave * 2 * kHalf];
            if (lane < kHalf) {
                blk[2 * lane] = __builtin_amdgcn_cosf(ub);
                blk[2 * lane + 1] = __builtin_amdgcn_sinf(ub);
            }
            // the wave's own LDS writes complete before its later LDS reads; the fence keeps
            // the compiler from moving the reads above the writes
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
            __builtin_amdgcn_wave_barrier();
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
            for (int c = 0; c < kChunks; ++c) {
                const bool kept = c == kChunks - 1 || ((keep >> (8 * c)) & 0xFFull) != 0;
                if (kept) {
                    const float* row = &s_colcs[col * kCStride + 16 * c];
                    const float* brow = blk + 16 * c;
                    float cs8[8], sn8[8];
#pragma unroll
                    for (int q4 = 0; q4 < 4; ++q4) {
                        const float4 v = *reinterpret_cast<const float4*>(row + 4 * q4);  // pairs 2q4, 2q4+1
                        const float4 w = *reinterpret_cast<const float4*>(brow + 4 * q4);
#pragma unroll
                        for (int j = 0; j < 2; ++j) {
                            const int e = 2 * q4 + j;
                            const float cB = j ? w.z : w.x, sB = j ? w.w : w.y;
                            const float cC = j ? v.z : v.x, sC = j ? v.w : v.y;
                            cs8[e] = __builtin_fmaf(cB, cC, -sB * sC);
                            sn8[e] = __builtin_fmaf(sB, cC, cB * sC);
                        }
                    }
                    kf[c] = rope::rotate_cs(kf[c], rope::other_half(kf[c], hh), hh, cs8, sn8);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        // QK (lowest frequencies first; one MFMA site per chunk)
        f32x16_t sacc;
#pragma unroll
        for (int c = kChunks - 1; c >= 0; --c) {
            const uint32_t fc = uint32_t(full >> (8 * c)) & 0xFFu;
            if (c == kChunks - 1) {
                sacc = mfma(kf[c], keep_pairs(qf[c], fc), zero16());
            } else if (fc) {
                u32x4_t qb = qf[c];
                if (fc != 0xFFu) qb = keep_pairs(qb, fc);
                sacc = mfma(kf[c], qb, sacc);
            }
        }
        // pairs whose window ends inside the block (register v: token t0 + off(v) + 4 hh),
        // grouped by chunk and threshold: one MFMA per group
        uint64_t part = keep & ~full;
        while (part) {
            const int r = __builtin_ctzll(part);
            const int c = r >> 3;
            const int wr = __builtin_amdgcn_readlane(my_w, r);
            const uint64_t grp = __ballot(my_w == wr) & part & (0xFFull << (8 * c));
            part &= ~grp;
            u32x4_t kfc = kf[0], qfc = qf[0];
#pragma unroll
            for (int cc = 1; cc < kChunks; ++cc)
                if (cc == c) {
                    kfc = kf[cc];
                    qfc = qf[cc];
                }
            const f32x16_t t = mfma(kfc, keep_pairs(qfc, uint32_t(grp >> (8 * c))), zero16());
            const int thr = q_pos - t0 - 4 * hh - wr;  // keep iff off(v) >= thr
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int off = 8 * (v / 4) + (v % 4);
                sacc[v] += off >= thr ? t[v] : 0.f;
            }
        }
        if constexpr (kRot) {
            // the next block's K (past the split's last block the current block is loaded
            // again, so that the loads in flight do not depend on the path)
            const int tn = t0 + 32 * kWaves < t_end ? t0 + 32 * kWaves : t0;
            B = locate(tn);
            load_k(B, tn);
        }
        // tokens past the split's end
        if (t0 + 32 > t_end) {
            const int bound = t_end - t0 - 4 * hh;
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int off = 8 * (v / 4) + (v % 4);
                if (off >= bound) sacc[v] = -INFINITY;
            }
        }

        // online softmax per head column
        float mx = -INFINITY;
#pragma unroll
        for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sacc[v]);
        // the two lane halves of a column share m_run and sc > 0: some lane's half max
        // passes the threshold exactly when some column max does, so the halves exchange
        // their maxima only when the running max is raised
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
            for (int i = 0; i < kDB; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v) oacc[i][v] *= alpha;
        }
        u32x4_t pb[2];
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const float a = exp2_fast(__builtin_fmaf(sacc[8 * ks + 2 * t], sc, m_neg));
                const float c2 = exp2_fast(__builtin_fmaf(sacc[8 * ks + 2 * t + 1], sc, m_neg));
                l_run += a;
                l_run += c2;
                bf16x2_t two;
                two[0] = (__bf16)a;
                two[1] = (__bf16)c2;
                pb[ks][t] = __builtin_bit_cast(uint32_t, two);
            }
        }
        // PV
#pragma unroll
        for (int ks = 0; ks < 2; ++ks)
#pragma unroll
            for (int i = 0; i < kDB; ++i) oacc[i] = mfma(vf[ks][i], pb[ks], oacc[i]);
    }

    // ---- combine the four waves' states (in wave order, so the result is
    // deterministic) and write the split's partial
    const float l_lane = l_run + __shfl_xor(l_run, 32);
    if (hh == 0) {
        red_m[wave][col] = m_run;
        red_l[wave][col] = l_lane;
    }
    __syncthreads();
    float m_all = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) m_all = fmaxf(m_all, red_m[w][col]);
    const float f = m_run == -INFINITY ? 0.f : exp2_fast(m_run - m_all);
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
        if (wave == w && head_ok) {
#pragma unroll
            for (int i = 0; i < kDB; ++i)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    float& dst = red_o[col][32 * i + 8 * (v / 4) + 4 * hh + (v % 4)];
                    dst = (w == 0 ? 0.f : dst) + oacc[i][v] * f;
                }
        }
        __syncthreads();
    }
    for (int e = tid; e < NH * D; e += kWaves * 64) {
        const int h = e / D, x = e % D;
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < kWaves; ++w) M = fmaxf(M, red_m[w][h]);
        float L = 0.f;
        if (M != -INFINITY) {
#pragma unroll
            for (int w = 0; w < kWaves; ++w)
                if (red_m[w][h] != -INFINITY) L += red_l[w][h] * exp2_fast(red_m[w][h] - M);
        }
        const int64_t slot = p.n_k_rows != nullptr ? slot0 + h : slot0 + int64_t(h) * p.splits;
        if (x == 0) {
            p.ws_m[slot] = M;
            p.ws_l[slot] = L;
        }
        p.ws_o[slot * D + x] = red_o[h][x];
    }
}

// Merge of the split partials of one (batch, head) and 32 output dims: 256 threads.
// The weights take one state per thread; the output sums take 8 quads of 4 dims x 32
// state lanes, each lane reading 16 bytes per state, so that all of a thread's loads
// can be in flight at once.
template <int D>
__global__ __launch_bounds__(256) void decode_merge_kernel(const DecodeParams p) {
    __shared__ float s_w[kDecodeMaxSplits];  // split weights exp2(m_s - M)
    __shared__ float s_red[8];     // per-wave max, then per-wave sum
    __shared__ float s_o[32][33];  // output partial sums of the 32 state lanes
    const int bh = blockIdx.x;  // b * h_q + hq
    const int d0 = 32 * blockIdx.y;
    const int tid = threadIdx.x;
    // partial state s of this (row, head) at slot base + s * stride: a uniform batch
    // has p.splits of them per head; a ragged row has the items the plan gave it
    int64_t base = int64_t(bh) * p.splits, stride = 1;
    int count = p.splits;
    if (p.n_k_rows != nullptr) {
        const int b = bh / p.h_q;
        // (the clamps only restate what the plan guarantees: items < splits + batch)
        const int first = min(max(p.ws_plan[b], 0), p.splits + p.batch);
        count = min(min(max(p.ws_plan[b + 1] - first, 0), kDecodeMaxSplits),
                    p.splits + p.batch - first);
        base = int64_t(first) * p.h_q + bh % p.h_q;
        stride = p.h_q;
    }
    const int wave = tid >> 6;
    float M = -INFINITY;
    for (int s = tid; s < count; s += 256) M = fmaxf(M, p.ws_m[base + s * stride]);
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
    if ((tid & 63) == 0) s_red[wave] = M;
    __syncthreads();
    M = fmaxf(fmaxf(s_red[0], s_red[1]), fmaxf(s_red[2], s_red[3]));
    float L = 0.f;
    for (int s = tid; s < count; s += 256) {
        const float ms = p.ws_m[base + s * stride];
        const float w = ms == -INFINITY ? 0.f : exp2_fast(ms - M);  // split with no causal key
        s_w[s] = w;
        L += p.ws_l[base + s * stride] * w;
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) L += __shfl_xor(L, o);
    if ((tid & 63) == 0) s_red[4 + wave] = L;
    __syncthreads();  // also publishes s_w
    L = (s_red[4] + s_red[5]) + (s_red[6] + s_red[7]);
    const int q = tid & 7, sl = tid >> 3;  // dims d0 + 4q .. d0 + 4q + 3, state lane sl
    float4 O = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll 8
    for (int s = sl; s < count; s += 32) {
        const float w = s_w[s];
        const float4 v = *reinterpret_cast<const float4*>(p.ws_o + (base + s * stride) * D + d0 + 4 * q);
        O.x += w * v.x;
        O.y += w * v.y;
        O.z += w * v.z;
        O.w += w * v.w;
    }
    s_o[sl][4 * q] = O.x;
    s_o[sl][4 * q + 1] = O.y;
    s_o[sl][4 * q + 2] = O.z;
    s_o[sl][4 * q + 3] = O.w;
    __syncthreads();
    if (tid < 32) {
        const int x = tid;
        float acc = 0.f;
#pragma unroll
        for (int k = 0; k < 32; ++k) acc += s_o[k][x];
        // a ragged row without keys has an empty softmax: O = 0, LSE = -inf
        const bool empty = !(L > 0.f);
        p.o[int64_t(bh) * D + d0 + x] = __builtin_bit_cast(uint16_t, (__bf16)(empty ? 0.f : acc / L));
        if (blockIdx.y == 0 && tid == 0) p.lse[bh] = empty ? -INFINITY : M * 0.69314718055994531f + logf(L);
    }
}

template <int D>
__global__ __launch_bounds__(256) void pack_kcache_kernel(const PackParams p) {
    constexpr int kChunks = D / 16;
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
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
        const u32x4 lo = *reinterpret_cast<const u32x4*>(src + 8 * c);
        const u32x4 hi = *reinterpret_cast<const u32x4*>(src + D / 2 + 8 * c);
        uint16_t* dst = p.dst + (((int64_t(b) * p.h_kv + g) * kChunks + c) * p.cache_tokens +
                                 p.pos0 + t) * 16;
        *reinterpret_cast<u32x4*>(dst) = lo;
        *reinterpret_cast<u32x4*>(dst + 8) = hi;
    }
}

// V blocks: one thread per (batch, kv head, touched 16-token block, dim); slot
// 8h + e of the row holds token 8*(e/4) + 4h + e%4 of the block.  Slots of
// tokens outside pos0 .. pos0 + n_k - 1 keep their contents (or become 0 past the
// source when zero_tail is set).
template <int D>
__global__ __launch_bounds__(256) void pack_vcache_kernel(const PackParams p) {
    const int blk0 = p.pos0 / 16;
    const int nblk = (p.pos0 + p.n_k + 15) / 16 - blk0;  // blocks touched
    const int cache_blk = (p.cache_tokens + 15) / 16;
    const int64_t total = int64_t(p.batch) * p.h_kv * nblk * D;
    for (int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x; idx < total;
         idx += int64_t(gridDim.x) * 256) {
        const int x = int(idx % D);
        int64_t r = idx / D;
        const int blk = blk0 + int(r % nblk);
        r /= nblk;
        const int g = int(r % p.h_kv);
        const int b = int(r / p.h_kv);
        uint16_t* dst = p.dst + ((int64_t(b) * p.h_kv + g) * cache_blk + blk) * int64_t(D) * 16 +
                        int64_t(x) * 16;
#pragma unroll
        for (int pos = 0; pos < 16; ++pos) {
            const int h = pos >> 3, e = pos & 7;
            const int t = 16 * blk + 8 * (e >> 2) + 4 * h + (e & 3) - p.pos0;  // source token
            if (t >= 0 && t < p.n_k)
                dst[pos] = p.src[((int64_t(b) * p.n_k + t) * p.h_kv + g) * D + x];
            else if (t >= p.n_k && p.zero_tail)
                dst[pos] = uint16_t(0);
        }
    }
}

// Paged append: one thread per (batch, new token, kv head, 8-dim piece); K pieces
// go to the token's chunk stream in its page, V elements to the slots of the
// token's 16-token block in its page (slot 8h + e holds token 8(e/4) + 4h + e%4).
template <int D>
__global__ __launch_bounds__(256) void append_paged_kernel(const AppendPagedParams p) {
    constexpr int kChunks = D / 16;
    constexpr int kPieces = D / 8;  // 8-dim pieces of one (token, head) row
    typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
    const int64_t total = int64_t(p.batch) * p.n_new * p.h_kv * kPieces;
    for (int64_t idx = int64_t(blockIdx.x) * 256 + threadIdx.x; idx < total;
         idx += int64_t(gridDim.x) * 256) {
        const int pc = int(idx % kPieces);
        int64_t r = idx / kPieces;
        const int g = int(r % p.h_kv);
        r /= p.h_kv;
        const int t = int(r % p.n_new);
        const int b = int(r / p.n_new);
        const int pos = p.pos0 + t;
        const int page = p.block_table[int64_t(b) * p.max_pages + pos / p.page_tokens];
        if (page < 0 || page >= p.num_pages) continue;
        const int slot = pos % p.page_tokens;
        const int64_t src = ((int64_t(b) * p.n_new + t) * p.h_kv + g) * D + 8 * pc;
        // K: piece pc = dims [8 pc, 8 pc + 8) is half (pc >= kChunks) of chunk pc % kChunks
        const int c = pc % kChunks, half = pc / kChunks;
        uint16_t* kd = p.k_pages + (((int64_t(page) * p.h_kv + g) * kChunks + c) * p.page_tokens +
                                    slot) * 16 + 8 * half;
        *reinterpret_cast<u32x4*>(kd) = *reinterpret_cast<const u32x4*>(p.k_src + src);
        // V: dims 8 pc .. 8 pc + 7 of this token, one slot each
        const int e16 = slot % 16;  // token within its 16-token block
        const int h = (e16 % 8) / 4, e = (e16 / 8) * 4 + e16 % 4;  // slot 8h + e
        uint16_t* vd = p.v_pages + ((int64_t(page) * p.h_kv + g) * (p.page_tokens / 16) + slot / 16) *
                                       int64_t(D) * 16 + 8 * h + e;
#pragma unroll
        for (int x = 0; x < 8; ++x) vd[int64_t(8 * pc + x) * 16] = p.v_src[src + x];
    }
}

template <int D>
hipError_t launch_decode_d(const DecodeParams& p, hipStream_t stream) {
    // ragged: one workgroup per possible work item (at most p.splits + batch)
    const bool ragged = p.n_k_rows != nullptr;
    const dim3 grid(unsigned(ragged ? p.splits + p.batch : p.splits),
                    unsigned(p.h_kv * (p.group / p.heads_per_block)), unsigned(ragged ? 1 : p.batch));
    if (p.rotate)
        hipLaunchKernelGGL((decode_split_kernel<D, true>), grid, dim3(kWaves * 64), 0, stream, p);
    else
        hipLaunchKernelGGL((decode_split_kernel<D, false>), grid, dim3(kWaves * 64), 0, stream, p);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(decode_merge_kernel<D>, dim3(unsigned(p.batch * p.h_q), unsigned(D / 32)),
                       dim3(256), 0, stream, p);
    return hipGetLastError();
}

unsigned pack_blocks(int64_t total) {
    int64_t blocks = (total + 255) / 256;
    return unsigned(blocks > 65536 ? 65536 : blocks);
}

}  // namespace

hipError_t launch_decode(const DecodeParams& p, int head_dim, hipStream_t stream) {
    if (p.splits < 1 || p.splits > kDecodeMaxSplits) return hipErrorInvalidValue;
    if (p.heads_per_block < 1 || p.heads_per_block > kDecodeMaxHeads ||
        p.group % p.heads_per_block != 0)
        return hipErrorInvalidValue;
    if (p.n_k_rows == nullptr &&
        (int64_t(p.splits) * p.split_tokens < p.n_valid || p.split_tokens % kDecodeTokenStep != 0))
        return hipErrorInvalidValue;
    if (p.n_k_rows != nullptr && (p.q_pos_rows == nullptr || p.ws_plan == nullptr ||
                                  p.splits > kDecodeMaxSplits - 1))
        return hipErrorInvalidValue;
    (void)hipGetLastError();
    return head_dim == 64 ? launch_decode_d<64>(p, stream) : launch_decode_d<128>(p, stream);
}

// The decode workspace of atf_decode_noalloc: a file-scope device array, so that
// callers that cannot allocate (graph capture, allocation-free serving loops) need
// no workspace.  Every device the library runs on holds its own copy for the life
// of the process; calls on one device share it (the last call's partial states stay
// in it), so such calls must not overlap.  In host code `scratch` names a host-side
// stand-in, never the device memory: its device address comes from
// hipGetSymbolAddress, once per device, with that device current.
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxScratchDevices] = {};
}  // namespace

hipError_t noalloc_scratch(void** out) {
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_addr[dev] == nullptr) {
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (ptr == nullptr) return hipErrorInvalidSymbol;
        g_scratch_addr[dev] = ptr;
    }
    *out = g_scratch_addr[dev];
    return hipSuccess;
}

hipError_t launch_pack_kcache(const PackParams& p, int head_dim, hipStream_t stream) {
    const int64_t total = int64_t(p.batch) * p.n_k * p.h_kv * (head_dim / 16);
    (void)hipGetLastError();
    if (head_dim == 64)
        hipLaunchKernelGGL(pack_kcache_kernel<64>, dim3(pack_blocks(total)), dim3(256), 0, stream, p);
    else
        hipLaunchKernelGGL(pack_kcache_kernel<128>, dim3(pack_blocks(total)), dim3(256), 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_append_paged(const AppendPagedParams& p, int head_dim, hipStream_t stream) {
    const int64_t total = int64_t(p.batch) * p.n_new * p.h_kv * (head_dim / 8);
    (void)hipGetLastError();
    if (head_dim == 64)
        hipLaunchKernelGGL(append_paged_kernel<64>, dim3(pack_blocks(total)), dim3(256), 0, stream, p);
    else
        hipLaunchKernelGGL(append_paged_kernel<128>, dim3(pack_blocks(total)), dim3(256), 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_pack_vcache(const PackParams& p, int head_dim, hipStream_t stream) {
    const int64_t total = int64_t(p.batch) * p.h_kv *
                          ((p.pos0 + p.n_k + 15) / 16 - p.pos0 / 16) * head_dim;
    (void)hipGetLastError();
    if (head_dim == 64)
        hipLaunchKernelGGL(pack_vcache_kernel<64>, dim3(pack_blocks(total)), dim3(256), 0, stream, p);
    else
        hipLaunchKernelGGL(pack_vcache_kernel<128>, dim3(pack_blocks(total)), dim3(256), 0, stream, p);
    return hipGetLastError();
}

}  // namespace atf
