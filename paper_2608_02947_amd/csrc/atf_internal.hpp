// Internal declarations shared by the host side of libatf.so and its kernels.
// Not part of the public ABI (include/atf.h is).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace atf {

constexpr int kMaxPairs = 64;     // d/2 for d = 128
constexpr int kChunkPairs = 8;    // pairs per QK K-step and per decode K-cache chunk
constexpr int kMaxChunks = kMaxPairs / kChunkPairs;

// Window table in the form every kernel consumes: per pair the integer threshold
// W_r (keep the pair's term at distance z iff z <= W_r), and per chunk of
// kChunkPairs consecutive pairs the smallest and largest threshold.
struct WindowTable {
    int32_t W[kMaxPairs];
    int32_t chunk_min[kMaxChunks];
    int32_t chunk_max[kMaxChunks];
};

struct PrefillParams {
    const uint16_t* q;   // [B][n_q][h_q][d]
    const uint16_t* k;   // [B][h_kv][d/16][cache_tokens][16] (pair-chunk-major)
    const uint16_t* v;   // [B][h_kv][ceil(cache_tokens/16)][d][16] (see atf_pack_vcache)
    uint16_t* o;         // [B][n_q][h_q][d]
    float* lse;          // [B][h_q][n_q]
    int32_t batch, n_q, n_k, q_pos0, h_q, h_kv, group;
    int32_t cache_tokens;  // tokens each cache entry is allocated for (>= n_k)
    int32_t pos_per_tile;  // query positions per workgroup (rows = positions x group)
    int32_t n_qtiles;
    int32_t mono;        // thresholds non-decreasing and the last chunk kept at every distance
    float scale_log2;    // softmax scale * log2(e)
    WindowTable win;
};

// Prefill with RoPE at read time: q and the K cache hold unrotated vectors, rotated
// in the kernel as DecodeParams describes. A type of its own, so that the kernels
// of pre-rotated caches keep their argument block.
struct PrefillRotParams : PrefillParams {
    uint32_t rope_rho_hi[kMaxPairs];
    uint32_t rope_rho_lo[kMaxPairs];
};

struct DecodeParams {
    const uint16_t* q;       // [B][h_q][d]
    const uint16_t* kpcm;    // [B][h_kv][d/16][cache_tokens][16]
    const uint16_t* vpk;     // [B][h_kv][ceil(cache_tokens/16)][d][16] (see atf_pack_vcache)
    uint16_t* o;             // [B][h_q][d]
    float* lse;              // [B][h_q]
    float* ws_m;             // [B][h_q][splits]   running max (log2 domain)
    float* ws_l;             // [B][h_q][splits]   normaliser
    float* ws_o;             // [B][h_q][splits][d] unnormalised output
    int32_t batch, n_k, q_pos, h_q, h_kv, group;
    int32_t cache_tokens;     // tokens each cache entry is allocated for (>= n_k)
    int32_t heads_per_block;  // query heads handled by one workgroup (divides group, <= 32)
    int32_t n_valid;          // keys 0 .. n_valid - 1 are causal
    const int32_t* n_k_rows;  // ragged batch: device [B] keys of each row (clamped to
                              // [0, n_k]), or nullptr: every row has n_k keys
    const int32_t* q_pos_rows;  // ragged batch: device [B] query position of each row
                                // (clamped to [0, 2^31 - 2]), or nullptr: q_pos
    const int32_t* block_table;  // paged caches: device [B][max_pages] page of each row's
                                 // page_tokens-token span (clamped to [0, num_pages)),
                                 // or nullptr: contiguous caches
    int32_t max_pages, num_pages, page_tokens;
    int32_t* ws_plan;         // ragged batch: [B + 1] index of each row's first work item
                              // (written by the split kernel for the merge), else unused
    int32_t splits;           // uniform batch: splits per row; ragged batch: work items the
                              // batch's keys are spread over (a row adds at most one more)
    int32_t split_tokens;     // uniform batch: tokens per split (multiple of the workgroup's
                              // token step); ragged batch: unused (derived on the device)
    float scale_log2;
    WindowTable win;
    // RoPE at read time: q and the K cache hold unrotated vectors; pair r of a vector
    // at position pos is rotated by pos * theta_r, with rho_r = theta_r / (2 pi) mod 1
    // as a 0.64 fixed-point fraction (hi and lo words)
    int32_t rotate;
    uint32_t rope_rho_hi[kMaxPairs];
    uint32_t rope_rho_lo[kMaxPairs];
};

struct AppendPagedParams {
    const uint16_t* k_src;     // [B][n_new][h_kv][d]: tokens pos0 .. pos0 + n_new - 1
    const uint16_t* v_src;
    uint16_t* k_pages;         // [num_pages][h_kv][d/16][page_tokens][16]
    uint16_t* v_pages;         // [num_pages][h_kv][page_tokens/16][d][16]
    const int32_t* block_table;  // [B][max_pages]
    int32_t batch, n_new, pos0, h_kv, max_pages, num_pages, page_tokens;
};

// The paged append with RoPE on the way in (rotate.hip): AppendPagedParams' fields, and
// the rotation's 0.64 fixed-point frequencies.
struct RotatePagedParams {
    AppendPagedParams a;
    uint32_t rope_rho_hi[kMaxPairs];
    uint32_t rope_rho_lo[kMaxPairs];
};

struct PackParams {
    const uint16_t* src;  // [B][n_k][h_kv][d]: tokens pos0 .. pos0 + n_k - 1
    uint16_t* dst;        // K: [B][h_kv][d/16][cache_tokens][16];
                          // V: [B][h_kv][ceil(cache_tokens/16)][d][16]
    int32_t batch, n_k, h_kv;
    int32_t pos0;          // cache position of the first source token
    int32_t cache_tokens;  // capacity of dst
    int32_t zero_tail;     // V: write zeros to the slots of the touched blocks past the source
};

// One pass of RoPE into a pair-chunk-major K cache (rotate.hip).  Whole cache: key t
// of every (batch, kv head) at position t, tokens 0 .. n_k - 1, src in the cache layout.
// Append: src [B][n_k][h_kv][d] (as the projections give it), token t written at cache
// position pos0 + t and turned to that position.
struct RotateParams {
    const uint16_t* src;   // [B][h_kv][d/16][cache_tokens][16] (whole) or [B][n_k][h_kv][d] (append)
    uint16_t* dst;         // [B][h_kv][d/16][cache_tokens][16]; only the tokens named are written
    int32_t batch, n_k, h_kv, cache_tokens;
    int32_t pos0;          // append: cache position of the first source token
    uint32_t rope_rho_hi[kMaxPairs];
    uint32_t rope_rho_lo[kMaxPairs];
};

// Kernel launchers (prefill.hip, decode.hip, rotate.hip).  Return the HIP error of the launch.
hipError_t launch_prefill(const PrefillParams& p, int head_dim, hipStream_t stream);
hipError_t launch_prefill_rotating(const PrefillRotParams& p, int head_dim, hipStream_t stream);
hipError_t launch_decode(const DecodeParams& p, int head_dim, hipStream_t stream);
hipError_t launch_pack_kcache(const PackParams& p, int head_dim, hipStream_t stream);
hipError_t launch_pack_vcache(const PackParams& p, int head_dim, hipStream_t stream);
hipError_t launch_append_paged(const AppendPagedParams& p, int head_dim, hipStream_t stream);
hipError_t launch_rotate_kcache(const RotateParams& p, int head_dim, hipStream_t stream);
hipError_t launch_append_rotated_k(const RotateParams& p, int head_dim, hipStream_t stream);
hipError_t launch_append_paged_rotated(const RotatePagedParams& p, int head_dim, hipStream_t stream);

// Decode split plan of a uniform batch: number of KV splits per (batch, kv head).
int32_t decode_splits(int32_t batch, int32_t h_kv, int64_t n_k);
// Work items of a ragged batch (per column of `cols` = kv heads x head subgroups).
int32_t decode_ragged_items(int32_t cols);
// Tokens handled per decode workgroup iteration (the split granularity).
constexpr int32_t kDecodeTokenStep = 128;
// Largest split count the merge kernel accepts.
constexpr int32_t kDecodeMaxSplits = 4096;
// Query heads one decode workgroup handles at most (columns of its MFMA tiles).
constexpr int32_t kDecodeMaxHeads = 32;
// Size of the library's own decode scratch array (decode.hip), the workspace of
// atf_decode_noalloc; equal to ATF_DECODE_NOALLOC_SCRATCH_BYTES of atf.h.
constexpr size_t kNoAllocScratchBytes = size_t(16) << 20;
// Device address of that array on the current device, resolved once per device
// (hipGetSymbolAddress) and kept for the life of the process.
hipError_t noalloc_scratch(void** out);

}  // namespace atf
