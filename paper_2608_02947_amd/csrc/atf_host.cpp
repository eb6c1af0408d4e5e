// Host side of libatf.so: argument validation, the window table, the exact
// retained-term count, and dispatch to the gfx950 kernels.  See include/atf.h.
#include "atf.h"

#include <cmath>
#include <cstdarg>
#include <new>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <string>

#include "atf_internal.hpp"

namespace {

thread_local std::string g_last_error;

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return code;
}

constexpr int64_t kPosLimit = 2147483647;  // positions and thresholds are int32 on the device

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// W_r = floor(w_r), clamped to [0, 2^31 - 1], in fp64.  The default window is
// w_r = k * lambda_r with lambda_r = 2*pi/theta_r (eq:lambda, eq:window); with
// `family` set, w_r = min(max(k_r * lambda_r^gamma + a (r+1)/(d/2), beta), cap)
// (App. A eq:family).  A position-free pair (theta_r == 0) is never pruned.
// Works for any even d <= 2 * max_pairs.
int window_thresholds(const atf_window* w, int32_t* out, int max_pairs) {
    if (w == nullptr || out == nullptr) return fail(ATF_EINVAL, "window: NULL pointer");
    const int d = w->head_dim;
    if (d < 2 || d % 2 != 0 || d / 2 > max_pairs)
        return fail(ATF_EINVAL, "window: head_dim %d must be even, >= 2 and <= %d", d,
                    2 * max_pairs);
    const bool fam = w->family != 0;
    if (fam ? !(w->k >= 0.0) : !(w->k > 0.0))
        return fail(ATF_EINVAL, "window: k must be %s (got %g)", fam ? ">= 0" : "> 0", w->k);
    if (w->inv_freq == nullptr && !(w->rope_base > 1.0 && std::isfinite(w->rope_base)))
        return fail(ATF_EINVAL, "window: rope_base must be finite and > 1 (got %g)",
                    w->rope_base);
    if (fam) {
        if (!std::isfinite(w->gamma))
            return fail(ATF_EINVAL, "window: gamma must be finite (got %g)", w->gamma);
        if (!(w->a >= 0.0) || !std::isfinite(w->a))
            return fail(ATF_EINVAL, "window: a must be finite and >= 0 (got %g)", w->a);
        if (!(w->beta >= 0.0) || !std::isfinite(w->beta))
            return fail(ATF_EINVAL, "window: beta must be finite and >= 0 (got %g)", w->beta);
        if (!(w->cap >= 0.0))
            return fail(ATF_EINVAL, "window: cap must be >= 0 (got %g)", w->cap);
    }
    const double two_pi = 6.283185307179586476925286766559;
    for (int r = 0; r < d / 2; ++r) {
        double theta;
        if (w->inv_freq) {
            theta = w->inv_freq[r];
            if (!(theta >= 0.0) || std::isinf(theta))
                return fail(ATF_EINVAL, "window: inv_freq[%d] = %g must be finite and >= 0", r,
                            theta);
        } else {
            theta = std::pow(w->rope_base, -2.0 * r / d);
        }
        double width;
        if (theta == 0.0) {
            width = HUGE_VAL;  // no wavelength: every distance keeps the pair
        } else if (!fam) {
            width = w->k * (two_pi / theta);
        } else {
            const double kr = w->k_profile ? w->k_profile[r] : w->k;
            if (!(kr >= 0.0))
                return fail(ATF_EINVAL, "window: k_profile[%d] = %g must be >= 0", r, kr);
            width = kr * std::pow(two_pi / theta, w->gamma) + w->a * (r + 1) / (d / 2);
            if (std::isnan(width))
                return fail(ATF_EINVAL, "window: the width of pair %d is undefined (0 * inf)", r);
            width = std::fmin(std::fmax(width, w->beta), w->cap);
        }
        double t = std::floor(width);
        if (!(t < static_cast<double>(kPosLimit))) t = static_cast<double>(kPosLimit);
        if (t < 0.0) t = 0.0;
        out[r] = static_cast<int32_t>(t);
    }
    // Rounded slice (Sec. 3.3): at distance z the window keeps the suffix r >= rf(z)
    // of a non-decreasing table; rounding its length up to whole s-pair steps counted
    // from r = h - 1 keeps pair r iff the top pair of r's step is kept.
    const int h = d / 2, sp = w->slice_pairs;
    if (sp < 0 || sp > h)
        return fail(ATF_EINVAL, "window: slice_pairs %d must be in [0, d/2 = %d]", sp, h);
    if (sp > 1) {
        for (int r = 1; r < h; ++r)
            if (out[r] < out[r - 1])
                return fail(ATF_EINVAL,
                            "window: the rounded slice needs a table non-decreasing in r "
                            "(W[%d] = %d < W[%d] = %d)", r, out[r], r - 1, out[r - 1]);
        for (int r = 0; r < h; ++r) out[r] = out[h - 1 - sp * ((h - 1 - r) / sp)];
    }
    return ATF_OK;
}

int build_table(const atf_window* w, atf::WindowTable* t) {
    std::memset(t, 0, sizeof *t);
    int rc = window_thresholds(w, t->W, atf::kMaxPairs);
    if (rc != ATF_OK) return rc;
    const int pairs = w->head_dim / 2;
    for (int c = 0; c * atf::kChunkPairs < pairs; ++c) {
        int32_t lo = INT32_MAX, hi = 0;
        for (int e = 0; e < atf::kChunkPairs; ++e) {
            const int32_t x = t->W[c * atf::kChunkPairs + e];
            lo = x < lo ? x : lo;
            hi = x > hi ? x : hi;
        }
        t->chunk_min[c] = lo;
        t->chunk_max[c] = hi;
    }
    return ATF_OK;
}

using u128 = unsigned __int128;

// sum_{p=a}^{c} (p + 1), 0 <= a <= c
u128 sum_p_plus_1(int64_t a, int64_t c) {
    if (c < a) return 0;
    const u128 n = static_cast<u128>(c - a + 1);
    return n * static_cast<u128>(a + c + 2) / 2;
}

// Kept keys of one pair with threshold W, summed over rows p in [p0, p1]:
// per row, keys j in [max(0, p - W), min(p, n_k - 1)].
u128 pair_count(int64_t W, int64_t p0, int64_t p1, int64_t n_k) {
    u128 total = 0;
    // rows with p <= n_k - 1: min(p, W) + 1 keys
    {
        const int64_t a = p0, b = p1 < n_k - 1 ? p1 : n_k - 1;
        if (a <= b) {
            const int64_t c = b < W ? b : W;        // rows where p <= W: p + 1 keys
            total += sum_p_plus_1(a, c);
            const int64_t s = a > W + 1 ? a : W + 1;  // rows where p > W: W + 1 keys
            if (s <= b) total += static_cast<u128>(b - s + 1) * static_cast<u128>(W + 1);
        }
    }
    // rows with p >= n_k: n_k keys while p <= W, then n_k + W - p until it hits 0
    {
        const int64_t a = p0 > n_k ? p0 : n_k, b = p1;
        if (a <= b) {
            const int64_t c = b < W ? b : W;
            if (a <= c) total += static_cast<u128>(c - a + 1) * static_cast<u128>(n_k);
            const int64_t x = a > W + 1 ? a : W + 1;
            const int64_t y = b < n_k + W - 1 ? b : n_k + W - 1;
            if (x <= y) {
                const u128 n = static_cast<u128>(y - x + 1);
                total += n * static_cast<u128>(n_k + W) - n * static_cast<u128>(x + y) / 2;
            }
        }
    }
    return total;
}

}  // namespace

namespace atf {

int32_t decode_splits(int32_t batch, int32_t h_kv, int64_t n_k) {
    // enough workgroups to fill 256 CUs several times over, but never a split
    // shorter than one workgroup step
    const int64_t target_groups = 1024;
    int64_t s = (target_groups + int64_t(batch) * h_kv - 1) / (int64_t(batch) * h_kv);
    const int64_t max_s = (n_k + kDecodeTokenStep - 1) / kDecodeTokenStep;
    if (s > max_s) s = max_s;
    if (s > kDecodeMaxSplits) s = kDecodeMaxSplits;
    if (s < 1) s = 1;
    return static_cast<int32_t>(s);
}

int32_t decode_ragged_items(int32_t cols) {
    // the batch's keys are cut into about this many equal spans per column, whatever
    // the row lengths (measured on batches of 8 rows at d = 128 with 8 KV heads:
    // 2048 workgroups beat 1024 by 5-12 % and 4096 by 0-20 %, on rows of 4K-128K keys,
    // of 128K keys, and of one 128K row beside seven 1K rows)
    const int64_t target_groups = 2048;
    int64_t s = (target_groups + cols - 1) / cols;
    if (s > kDecodeMaxSplits - 1) s = kDecodeMaxSplits - 1;
    if (s < 1) s = 1;
    return static_cast<int32_t>(s);
}

}  // namespace atf

extern "C" {

const char* atf_last_error(void) { return g_last_error.c_str(); }

int atf_window_table(const atf_window* w, int32_t* W_out) {
    return window_thresholds(w, W_out, 1 << 20);
}

int atf_retention_profile(int32_t head_dim, int32_t kind, double k_hi, double k_lo,
                          double* k_out) {
    if (k_out == nullptr) return fail(ATF_EINVAL, "retention_profile: NULL output");
    if (head_dim < 2 || head_dim % 2 != 0)
        return fail(ATF_EINVAL, "retention_profile: head_dim %d must be even and >= 2", head_dim);
    if (!(k_hi >= 0.0) || !std::isfinite(k_hi) || !(k_lo >= 0.0) || !std::isfinite(k_lo))
        return fail(ATF_EINVAL, "retention_profile: k_hi, k_lo must be finite and >= 0");
    const int n = head_dim / 2;
    const double span = n > 1 ? double(n - 1) : 1.0;
    switch (kind) {
        case ATF_PROFILE_CONSTANT:
            for (int r = 0; r < n; ++r) k_out[r] = k_hi;
            return ATF_OK;
        case ATF_PROFILE_ARITHMETIC: {
            const double step = (k_hi - k_lo) / span;
            for (int r = 0; r < n; ++r) k_out[r] = k_hi - step * r;
            if (n > 1) k_out[n - 1] = k_lo;
            return ATF_OK;
        }
        case ATF_PROFILE_GEOMETRIC: {
            if (!(k_hi > 0.0) || !(k_lo > 0.0))
                return fail(ATF_EINVAL, "retention_profile: geometric needs k_hi, k_lo > 0");
            const double lr = std::log(k_lo / k_hi) / span;
            for (int r = 0; r < n; ++r) k_out[r] = k_hi * std::exp(lr * r);
            if (n > 1) k_out[n - 1] = k_lo;
            return ATF_OK;
        }
        default:
            return fail(ATF_EINVAL, "retention_profile: unknown kind %d", kind);
    }
}

int atf_count_terms(const atf_window* w, int64_t n_q, int64_t q_pos0, int64_t n_k,
                    uint64_t* retained, uint64_t* causal_cells) {
    if (retained == nullptr || causal_cells == nullptr)
        return fail(ATF_EINVAL, "count_terms: NULL output");
    if (n_q < 0 || q_pos0 < 0 || n_k < 0)
        return fail(ATF_EINVAL, "count_terms: n_q, q_pos0 and n_k must be >= 0");
    if (q_pos0 > INT64_MAX / 4 - n_q || n_k > INT64_MAX / 4)
        return fail(ATF_EINVAL, "count_terms: sizes too large");
    if (w == nullptr) return fail(ATF_EINVAL, "count_terms: NULL window");
    const int pairs = w->head_dim / 2;
    if (w->head_dim < 2 || w->head_dim % 2 || pairs > (1 << 20))
        return fail(ATF_EINVAL, "count_terms: bad head_dim %d", w->head_dim);
    int32_t* W = new (std::nothrow) int32_t[pairs];
    if (!W) return fail(ATF_EINVAL, "count_terms: out of host memory");
    int rc = window_thresholds(w, W, pairs);
    if (rc != ATF_OK) {
        delete[] W;
        return rc;
    }
    u128 ret = 0, cau = 0;
    if (n_q > 0 && n_k > 0) {
        const int64_t p0 = q_pos0, p1 = q_pos0 + n_q - 1;
        for (int r = 0; r < pairs; ++r) ret += pair_count(W[r], p0, p1, n_k);
        cau = pair_count(INT64_MAX / 8, p0, p1, n_k);  // every key kept
    }
    delete[] W;
    if (ret > static_cast<u128>(UINT64_MAX) || cau > static_cast<u128>(UINT64_MAX))
        return fail(ATF_EINVAL, "count_terms: count exceeds 64 bits");
    *retained = static_cast<uint64_t>(ret);
    *causal_cells = static_cast<uint64_t>(cau);
    return ATF_OK;
}

int32_t atf_kcache_chunk_pairs(int32_t head_dim) {
    return (head_dim == 64 || head_dim == 128) ? atf::kChunkPairs : 0;
}

namespace {

// RoPE at read time (q and the K cache unrotated): theta_r = rope_inv_freq[r] if given,
// else the window's frequencies (its inv_freq, or rope_base^(-2r/d)).
struct RopeArgs {
    bool rotate = false;
    const double* inv_freq = nullptr;
};

// rho_r = theta_r / (2 pi) mod 1 as a 0.64 fixed-point fraction, in extended precision
int rope_fractions(const char* fn, const atf_window* w, const double* inv_freq,
                   uint32_t* rho_hi, uint32_t* rho_lo) {
    const int d = w->head_dim;
    const long double two_pi = 6.283185307179586476925286766559L;
    for (int r = 0; r < d / 2; ++r) {
        double th;
        if (inv_freq != nullptr)
            th = inv_freq[r];
        else if (w->inv_freq != nullptr)
            th = w->inv_freq[r];
        else
            th = std::pow(w->rope_base, -2.0 * r / d);
        if (!(th >= 0.0) || std::isinf(th))
            return fail(ATF_EINVAL, "%s: rotation frequency %d = %g must be finite and >= 0", fn, r,
                        th);
        long double f = static_cast<long double>(th) / two_pi;
        f -= std::floor(f);
        long double scaled = std::ldexp(f, 64);
        uint64_t fx = scaled >= 18446744073709551615.0L ? UINT64_MAX : static_cast<uint64_t>(scaled);
        rho_hi[r] = static_cast<uint32_t>(fx >> 32);
        rho_lo[r] = static_cast<uint32_t>(fx);
    }
    return ATF_OK;
}

// Shared by atf_prefill (pre-rotated caches) and atf_prefill_unrotated (RoPE applied
// to q and each kept key pair as the kernel reads them).
int prefill_impl(const char* fn, const void* q, const void* k, const void* v, void* o, float* lse,
                 int32_t batch, int64_t n_q, int64_t n_k, int64_t q_pos0, int32_t h_q,
                 int32_t h_kv, int64_t cache_tokens, const atf_window* w, float softmax_scale,
                 void* hip_stream, const RopeArgs& rope) {
    if (w == nullptr) return fail(ATF_EINVAL, "%s: NULL window", fn);
    const int d = w->head_dim;
    if (d != 64 && d != 128)
        return fail(ATF_EUNSUPPORTED, "%s: head_dim %d not built (64 or 128)", fn, d);
    if (batch < 1 || n_q < 0 || n_k < 1 || q_pos0 < 0 || h_q < 1 || h_kv < 1)
        return fail(ATF_EINVAL,
                    "%s: need batch >= 1, n_q >= 0, n_k >= 1, q_pos0 >= 0, heads >= 1", fn);
    if (h_q % h_kv != 0)
        return fail(ATF_EINVAL, "%s: h_q %d not a multiple of h_kv %d", fn, h_q, h_kv);
    const int max_group = d == 64 ? 128 : 256;  // query rows of one prefill workgroup
    if (h_q / h_kv > max_group)
        return fail(ATF_EUNSUPPORTED, "%s: GQA ratio %d above %d not built for d = %d", fn,
                    h_q / h_kv, max_group, d);
    if (q_pos0 + n_q > kPosLimit || n_k > kPosLimit)
        return fail(ATF_EINVAL, "%s: positions must stay below 2^31 - 1", fn);
    if (cache_tokens == 0) cache_tokens = n_k;
    if (cache_tokens < n_k || cache_tokens > kPosLimit)
        return fail(ATF_EINVAL, "%s: cache_tokens %lld must be >= n_k %lld and < 2^31 - 1", fn,
                    (long long)cache_tokens, (long long)n_k);
    if (!std::isfinite(softmax_scale))
        return fail(ATF_EINVAL, "%s: softmax_scale must be finite", fn);
    atf::PrefillRotParams p{};
    int rc = build_table(w, &p.win);
    if (rc != ATF_OK) return rc;
    if (rope.rotate) {
        rc = rope_fractions(fn, w, rope.inv_freq, p.rope_rho_hi, p.rope_rho_lo);
        if (rc != ATF_OK) return rc;
    }
    if (n_q == 0) return ATF_OK;
    if (!q || !k || !v || !o || !lse) return fail(ATF_EINVAL, "%s: NULL tensor pointer", fn);
    if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(o, 16) ||
        !aligned(lse, 4))
        return fail(ATF_EINVAL, "%s: q/k/v/o must be 16-byte and lse 4-byte aligned", fn);
    const float scale = softmax_scale > 0.f ? softmax_scale : 1.0f / std::sqrt(float(d));
    p.q = static_cast<const uint16_t*>(q);
    p.k = static_cast<const uint16_t*>(k);
    p.v = static_cast<const uint16_t*>(v);
    p.o = static_cast<uint16_t*>(o);
    p.lse = lse;
    p.batch = batch;
    p.n_q = static_cast<int32_t>(n_q);
    p.n_k = static_cast<int32_t>(n_k);
    p.cache_tokens = static_cast<int32_t>(cache_tokens);
    p.q_pos0 = static_cast<int32_t>(q_pos0);
    p.h_q = h_q;
    p.h_kv = h_kv;
    p.group = h_q / h_kv;
    p.scale_log2 = scale * 1.4426950408889634f;
    const hipStream_t st = static_cast<hipStream_t>(hip_stream);
    const hipError_t e = rope.rotate ? atf::launch_prefill_rotating(p, d, st)
                                     : atf::launch_prefill(p, d, st);
    if (e != hipSuccess) return fail(ATF_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return ATF_OK;
}

}  // namespace

int atf_prefill(const void* q, const void* k, const void* v, void* o, float* lse,
                int32_t batch, int64_t n_q, int64_t n_k, int64_t q_pos0, int32_t h_q,
                int32_t h_kv, int64_t cache_tokens, const atf_window* w, float softmax_scale,
                void* hip_stream) {
    return prefill_impl("prefill", q, k, v, o, lse, batch, n_q, n_k, q_pos0, h_q, h_kv,
                        cache_tokens, w, softmax_scale, hip_stream, RopeArgs());
}

int atf_prefill_unrotated(const void* q, const void* k, const void* v, void* o, float* lse,
                          int32_t batch, int64_t n_q, int64_t n_k, int64_t q_pos0, int32_t h_q,
                          int32_t h_kv, int64_t cache_tokens, const atf_window* w,
                          const double* rope_inv_freq, float softmax_scale, void* hip_stream) {
    RopeArgs rope;
    rope.rotate = true;
    rope.inv_freq = rope_inv_freq;
    return prefill_impl("prefill_unrotated", q, k, v, o, lse, batch, n_q, n_k, q_pos0, h_q, h_kv,
                        cache_tokens, w, softmax_scale, hip_stream, rope);
}


namespace {
int check_pack(const char* what, const void* src, void* dst, int32_t batch, int64_t n_k,
               int32_t h_kv, int32_t head_dim, size_t dst_bytes) {
    if (head_dim != 64 && head_dim != 128)
        return fail(ATF_EUNSUPPORTED, "%s: head_dim %d not built", what, head_dim);
    if (batch < 1 || n_k < 1 || h_kv < 1 || n_k > kPosLimit)
        return fail(ATF_EINVAL, "%s: need batch >= 1, 1 <= n_k < 2^31, h_kv >= 1", what);
    if (!src || !dst) return fail(ATF_EINVAL, "%s: NULL pointer", what);
    if (!aligned(src, 16) || !aligned(dst, 16))
        return fail(ATF_EINVAL, "%s: pointers must be 16-byte aligned", what);
    const size_t src_bytes = size_t(batch) * size_t(n_k) * size_t(h_kv) * size_t(head_dim) * 2;
    const char* a = static_cast<const char*>(src);
    const char* b = static_cast<const char*>(dst);
    if (a < b + dst_bytes && b < a + src_bytes)
        return fail(ATF_EINVAL, "%s: buffers overlap", what);
    return ATF_OK;
}

size_t vcache_bytes(int32_t batch, int64_t n_k, int32_t h_kv, int32_t head_dim) {
    return size_t(batch) * size_t(h_kv) * size_t((n_k + 15) / 16) * 16 * size_t(head_dim) * 2;
}
}  // namespace

int atf_pack_kcache(const void* k_bshd, void* k_pcm, int32_t batch, int64_t n_k, int32_t h_kv,
                    int32_t head_dim, void* hip_stream) {
    const size_t bytes = size_t(batch) * size_t(n_k) * size_t(h_kv) * size_t(head_dim) * 2;
    int rc = check_pack("pack_kcache", k_bshd, k_pcm, batch, n_k, h_kv, head_dim, bytes);
    if (rc != ATF_OK) return rc;
    atf::PackParams p{static_cast<const uint16_t*>(k_bshd), static_cast<uint16_t*>(k_pcm), batch,
                      static_cast<int32_t>(n_k), h_kv, 0, static_cast<int32_t>(n_k), 0};
    hipError_t e = atf::launch_pack_kcache(p, head_dim, static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return fail(ATF_EHIP, "pack_kcache: launch failed: %s", hipGetErrorString(e));
    return ATF_OK;
}

int atf_rotate_kcache(const void* k_pcm, void* k_rot, int32_t batch, int64_t n_k, int32_t h_kv,
                      int64_t cache_tokens, const atf_window* w, const double* rope_inv_freq,
                      void* hip_stream) {
    const char* fn = "rotate_kcache";
    if (w == nullptr) return fail(ATF_EINVAL, "%s: NULL window", fn);
    const int d = w->head_dim;
    if (d != 64 && d != 128)
        return fail(ATF_EUNSUPPORTED, "%s: head_dim %d not built (64 or 128)", fn, d);
    if (batch < 1 || n_k < 1 || h_kv < 1 || n_k > kPosLimit)
        return fail(ATF_EINVAL, "%s: need batch >= 1, 1 <= n_k < 2^31, h_kv >= 1", fn);
    if (cache_tokens == 0) cache_tokens = n_k;
    if (cache_tokens < n_k || cache_tokens > kPosLimit)
        return fail(ATF_EINVAL, "%s: cache_tokens %lld must be >= n_k %lld and < 2^31 - 1", fn,
                    (long long)cache_tokens, (long long)n_k);
    if (int64_t(batch) * h_kv * (d / 16) > 65535)
        return fail(ATF_EUNSUPPORTED, "%s: batch * h_kv * d/16 above 65535", fn);
    atf::RotateParams p{};
    int rc = rope_fractions(fn, w, rope_inv_freq, p.rope_rho_hi, p.rope_rho_lo);
    if (rc != ATF_OK) return rc;
    if (!k_pcm || !k_rot) return fail(ATF_EINVAL, "%s: NULL pointer", fn);
    if (!aligned(k_pcm, 16) || !aligned(k_rot, 16))
        return fail(ATF_EINVAL, "%s: pointers must be 16-byte aligned", fn);
    const size_t bytes = size_t(batch) * size_t(h_kv) * size_t(d) * size_t(cache_tokens) * 2;
    const char* a = static_cast<const char*>(k_pcm);
    const char* b = static_cast<const char*>(k_rot);
    // in place (the same buffer) is allowed: each thread reads a record, then writes it
    if (a != b && a < b + bytes && b < a + bytes)
        return fail(ATF_EINVAL, "%s: buffers overlap", fn);
    p.src = static_cast<const uint16_t*>(k_pcm);
    p.dst = static_cast<uint16_t*>(k_rot);
    p.batch = batch;
    p.n_k = static_cast<int32_t>(n_k);
    p.h_kv = h_kv;
    p.cache_tokens = static_cast<int32_t>(cache_tokens);
    const hipError_t e = atf::launch_rotate_kcache(p, d, static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return fail(ATF_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return ATF_OK;
}

size_t atf_vcache_bytes(int32_t batch, int64_t n_k, int32_t h_kv, int32_t head_dim) {
    if (batch < 1 || n_k < 1 || h_kv < 1 || n_k > kPosLimit || (head_dim != 64 && head_dim != 128))
        return 0;
    return vcache_bytes(batch, n_k, h_kv, head_dim);
}

int atf_pack_vcache(const void* v_bshd, void* v_pack, int32_t batch, int64_t n_k, int32_t h_kv,
                    int32_t head_dim, void* hip_stream) {
    int rc = check_pack("pack_vcache", v_bshd, v_pack, batch, n_k, h_kv, head_dim,
                        (batch >= 1 && n_k >= 1 && h_kv >= 1 && n_k <= kPosLimit)
                            ? vcache_bytes(batch, n_k, h_kv, head_dim) : 0);
    if (rc != ATF_OK) return rc;
    atf::PackParams p{static_cast<const uint16_t*>(v_bshd), static_cast<uint16_t*>(v_pack), batch,
                      static_cast<int32_t>(n_k), h_kv, 0, static_cast<int32_t>(n_k), 1};
    hipError_t e = atf::launch_pack_vcache(p, head_dim, static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return fail(ATF_EHIP, "pack_vcache: launch failed: %s", hipGetErrorString(e));
    return ATF_OK;
}

namespace {
// Shared by atf_cache_append (keys stored as given) and atf_cache_append_rotated (keys
// turned to their cache positions on the way in: rope != nullptr).
int cache_append_impl(const char* fn, const void* k_new, const void* v_new, void* k_cache,
                      void* v_cache, int32_t batch, int64_t n_new, int64_t pos0, int32_t h_kv,
                      int32_t head_dim, int64_t cache_tokens, void* hip_stream,
                      const atf::RotateParams* rope) {
    if (head_dim != 64 && head_dim != 128)
        return fail(ATF_EUNSUPPORTED, "%s: head_dim %d not built", fn, head_dim);
    if (batch < 1 || h_kv < 1 || n_new < 0 || pos0 < 0 || cache_tokens < 1 ||
        cache_tokens > kPosLimit || pos0 > cache_tokens - n_new)
        return fail(ATF_EINVAL,
                    "%s: need batch >= 1, h_kv >= 1, n_new >= 0, pos0 >= 0, "
                    "1 <= cache_tokens < 2^31 and pos0 + n_new <= cache_tokens", fn);
    if (!k_new || !v_new || !k_cache || !v_cache)
        return fail(ATF_EINVAL, "%s: NULL pointer", fn);
    if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16))
        return fail(ATF_EINVAL, "%s: pointers must be 16-byte aligned", fn);
    const size_t row = size_t(h_kv) * size_t(head_dim) * 2;
    const char* bufs[4] = {static_cast<const char*>(k_new), static_cast<const char*>(v_new),
                           static_cast<const char*>(k_cache), static_cast<const char*>(v_cache)};
    const size_t sizes[4] = {size_t(batch) * size_t(n_new) * row, size_t(batch) * size_t(n_new) * row,
                             size_t(batch) * size_t(cache_tokens) * row,
                             vcache_bytes(batch, cache_tokens, h_kv, head_dim)};
    for (int i = 0; i < 4; ++i)
        for (int j = (i < 2 ? 2 : i + 1); j < 4; ++j)  // written buffers against all others
            if (bufs[i] < bufs[j] + sizes[j] && bufs[j] < bufs[i] + sizes[i])
                return fail(ATF_EINVAL, "%s: buffers overlap", fn);
    if (n_new == 0) return ATF_OK;
    const hipStream_t st = static_cast<hipStream_t>(hip_stream);
    atf::PackParams pk{static_cast<const uint16_t*>(k_new), static_cast<uint16_t*>(k_cache), batch,
                       static_cast<int32_t>(n_new), h_kv, static_cast<int32_t>(pos0),
                       static_cast<int32_t>(cache_tokens), 0};
    hipError_t e;
    if (rope != nullptr) {
        atf::RotateParams rp = *rope;
        rp.src = pk.src;
        rp.dst = pk.dst;
        rp.batch = batch;
        rp.n_k = pk.n_k;
        rp.h_kv = h_kv;
        rp.cache_tokens = pk.cache_tokens;
        rp.pos0 = pk.pos0;
        e = atf::launch_append_rotated_k(rp, head_dim, st);
    } else {
        e = atf::launch_pack_kcache(pk, head_dim, st);
    }
    if (e == hipSuccess) {
        atf::PackParams pv = pk;
        pv.src = static_cast<const uint16_t*>(v_new);
        pv.dst = static_cast<uint16_t*>(v_cache);
        e = atf::launch_pack_vcache(pv, head_dim, st);
    }
    if (e != hipSuccess) return fail(ATF_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return ATF_OK;
}
}  // namespace

int atf_cache_append(const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                     int32_t batch, int64_t n_new, int64_t pos0, int32_t h_kv, int32_t head_dim,
                     int64_t cache_tokens, void* hip_stream) {
    return cache_append_impl("cache_append", k_new, v_new, k_cache, v_cache, batch, n_new, pos0,
                             h_kv, head_dim, cache_tokens, hip_stream, nullptr);
}

int atf_cache_append_rotated(const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                             int32_t batch, int64_t n_new, int64_t pos0, int32_t h_kv,
                             int64_t cache_tokens, const atf_window* w, const double* rope_inv_freq,
                             void* hip_stream) {
    const char* fn = "cache_append_rotated";
    if (w == nullptr) return fail(ATF_EINVAL, "%s: NULL window", fn);
    const int d = w->head_dim;
    if (d != 64 && d != 128)
        return fail(ATF_EUNSUPPORTED, "%s: head_dim %d not built (64 or 128)", fn, d);
    atf::RotateParams rp{};
    const int rc = rope_fractions(fn, w, rope_inv_freq, rp.rope_rho_hi, rp.rope_rho_lo);
    if (rc != ATF_OK) return rc;
    return cache_append_impl(fn, k_new, v_new, k_cache, v_cache, batch, n_new, pos0, h_kv, d,
                             cache_tokens, hip_stream, &rp);
}

namespace {
size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

struct WsLayout {
    size_t off_plan, off_m, off_l, off_o, total;
};

// Partial states of `slots` (split or work item) x h_q heads, after `plan_ints` int32.
WsLayout ws_layout(size_t slots, int32_t h_q, int32_t head_dim, size_t plan_ints) {
    const size_t n = slots * size_t(h_q);
    WsLayout L;
    L.off_plan = 0;
    L.off_m = align_up(plan_ints * 4, 256);
    L.off_l = L.off_m + align_up(n * 4, 256);
    L.off_o = L.off_l + align_up(n * 4, 256);
    L.total = L.off_o + align_up(n * size_t(head_dim) * 4, 256);
    return L;
}

// query heads per decode workgroup: the largest divisor of the group up to 32
int32_t decode_heads_per_block(int32_t group) {
    for (int32_t c = atf::kDecodeMaxHeads; c >= 1; --c)
        if (group % c == 0) return c;
    return 1;
}

WsLayout uniform_layout(int32_t batch, int32_t h_q, int32_t h_kv, int64_t n_k, int32_t head_dim) {
    return ws_layout(size_t(batch) * size_t(atf::decode_splits(batch, h_kv, n_k)), h_q, head_dim, 0);
}

// ragged batch: at most items + batch work items (each row rounds its count up once)
WsLayout ragged_layout(int32_t batch, int32_t h_q, int32_t h_kv, int32_t head_dim) {
    const int32_t cols = h_kv * (h_q / h_kv / decode_heads_per_block(h_q / h_kv));
    const size_t items = size_t(atf::decode_ragged_items(cols)) + size_t(batch);
    return ws_layout(items, h_q, head_dim, size_t(batch) + 1);
}
}  // namespace

size_t atf_decode_workspace_bytes(int32_t batch, int32_t h_q, int32_t h_kv, int64_t n_k,
                                  int32_t head_dim) {
    if (batch < 1 || h_q < 1 || h_kv < 1 || h_q % h_kv || n_k < 1 || n_k > kPosLimit ||
        (head_dim != 64 && head_dim != 128))
        return 0;
    // covers both plans: uniform (atf_decode) and ragged (atf_decode_ragged / _paged)
    const size_t u = uniform_layout(batch, h_q, h_kv, n_k, head_dim).total;
    const size_t r = ragged_layout(batch, h_q, h_kv, head_dim).total;
    return u > r ? u : r;
}

}  // extern "C"

namespace {

// Shared by atf_decode (every row has n_k keys and its query at q_pos) and
// atf_decode_ragged (row b has n_k_rows[b] keys and its query at q_pos_rows[b],
// device arrays; n_k is then their upper bound and q_pos is unused).
struct PagedArgs {
    const int32_t* block_table = nullptr;
    int32_t max_pages = 0, num_pages = 0, page_tokens = 0;
};

int decode_impl(const char* fn, const void* q, const void* k_cache, const void* v_cache, void* o,
                float* lse, int32_t batch, int64_t n_k, int64_t q_pos, const int32_t* n_k_rows,
                const int32_t* q_pos_rows, int32_t h_q, int32_t h_kv, int64_t cache_tokens,
                const atf_window* w, float softmax_scale, void* workspace, size_t workspace_bytes,
                void* hip_stream, const PagedArgs& pg = PagedArgs(), const RopeArgs& rope = RopeArgs()) {
    const bool ragged = n_k_rows != nullptr || q_pos_rows != nullptr;
    if (w == nullptr) return fail(ATF_EINVAL, "%s: NULL window", fn);
    const int d = w->head_dim;
    if (d != 64 && d != 128)
        return fail(ATF_EUNSUPPORTED, "%s: head_dim %d not built (64 or 128)", fn, d);
    if (batch < 1 || n_k < 1 || q_pos < 0 || h_q < 1 || h_kv < 1)
        return fail(ATF_EINVAL, "%s: need batch >= 1, n_k >= 1, q_pos >= 0, heads >= 1", fn);
    if (h_q % h_kv != 0)
        return fail(ATF_EINVAL, "%s: h_q %d not a multiple of h_kv %d", fn, h_q, h_kv);
    if (q_pos >= kPosLimit || n_k > kPosLimit)
        return fail(ATF_EINVAL, "%s: positions must stay below 2^31 - 1", fn);
    if (cache_tokens == 0) cache_tokens = n_k;
    if (cache_tokens < n_k || cache_tokens > kPosLimit)
        return fail(ATF_EINVAL, "%s: cache_tokens %lld must be >= n_k %lld and < 2^31 - 1", fn,
                    (long long)cache_tokens, (long long)n_k);
    if (!std::isfinite(softmax_scale))
        return fail(ATF_EINVAL, "%s: softmax_scale must be finite", fn);
    atf::DecodeParams p{};
    int rc = build_table(w, &p.win);
    if (rc != ATF_OK) return rc;
    if (rope.rotate) {
        rc = rope_fractions(fn, w, rope.inv_freq, p.rope_rho_hi, p.rope_rho_lo);
        if (rc != ATF_OK) return rc;
        p.rotate = 1;
    }
    if (!q || !k_cache || !v_cache || !o || !lse)
        return fail(ATF_EINVAL, "%s: NULL tensor pointer", fn);
    if (ragged && (!n_k_rows || !q_pos_rows))
        return fail(ATF_EINVAL, "%s: NULL row-length or row-position array", fn);
    if (!aligned(q, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) || !aligned(o, 16) ||
        !aligned(lse, 4))
        return fail(ATF_EINVAL, "%s: q/k/v/o must be 16-byte and lse 4-byte aligned", fn);
    if (ragged && (!aligned(n_k_rows, 4) || !aligned(q_pos_rows, 4)))
        return fail(ATF_EINVAL, "%s: row arrays must be 4-byte aligned", fn);
    if (pg.block_table != nullptr && !aligned(pg.block_table, 4))
        return fail(ATF_EINVAL, "%s: block table must be 4-byte aligned", fn);
    const WsLayout L = ragged ? ragged_layout(batch, h_q, h_kv, d)
                              : uniform_layout(batch, h_q, h_kv, n_k, d);
    if (workspace == nullptr || workspace_bytes < L.total)
        return fail(ATF_EWORKSPACE, "%s: workspace of %zu bytes needed, %zu given", fn, L.total,
                    workspace == nullptr ? size_t(0) : workspace_bytes);
    if (!aligned(workspace, 16)) return fail(ATF_EINVAL, "%s: workspace must be 16-byte aligned", fn);
    const float scale = softmax_scale > 0.f ? softmax_scale : 1.0f / std::sqrt(float(d));
    const int32_t group = h_q / h_kv;
    const int32_t hpb = decode_heads_per_block(group);
    char* ws = static_cast<char*>(workspace);
    p.q = static_cast<const uint16_t*>(q);
    p.kpcm = static_cast<const uint16_t*>(k_cache);
    p.vpk = static_cast<const uint16_t*>(v_cache);
    p.o = static_cast<uint16_t*>(o);
    p.lse = lse;
    p.ws_plan = ragged ? reinterpret_cast<int32_t*>(ws + L.off_plan) : nullptr;
    p.ws_m = reinterpret_cast<float*>(ws + L.off_m);
    p.ws_l = reinterpret_cast<float*>(ws + L.off_l);
    p.ws_o = reinterpret_cast<float*>(ws + L.off_o);
    p.batch = batch;
    p.n_k = static_cast<int32_t>(n_k);
    p.cache_tokens = static_cast<int32_t>(cache_tokens);
    p.q_pos = static_cast<int32_t>(q_pos);
    p.h_q = h_q;
    p.h_kv = h_kv;
    p.group = group;
    p.heads_per_block = hpb;
    p.n_k_rows = n_k_rows;
    p.q_pos_rows = q_pos_rows;
    p.block_table = pg.block_table;
    p.max_pages = pg.max_pages;
    p.num_pages = pg.num_pages;
    p.page_tokens = pg.page_tokens;
    if (ragged) {
        // the work items are laid out on the device from the row arrays: the batch's
        // keys in about `splits` equal spans (multiples of the workgroup's token step)
        // per column, each row cut into whole spans of its own keys
        p.n_valid = static_cast<int32_t>(n_k);
        p.splits = atf::decode_ragged_items(h_kv * (group / hpb));
        p.split_tokens = 0;
    } else {
        const int64_t last = q_pos < n_k - 1 ? q_pos : n_k - 1;
        p.n_valid = static_cast<int32_t>(last + 1);
        const int32_t splits = atf::decode_splits(batch, h_kv, n_k);
        p.splits = splits;
        const int64_t per = (p.n_valid + splits - 1) / splits;
        const int64_t step_tokens = (per + atf::kDecodeTokenStep - 1) / atf::kDecodeTokenStep *
                                    atf::kDecodeTokenStep;
        if (step_tokens * splits >= kPosLimit)
            return fail(ATF_EINVAL, "%s: cache too long for the split plan", fn);
        p.split_tokens = static_cast<int32_t>(step_tokens);
    }
    p.scale_log2 = scale * 1.4426950408889634f;
    hipError_t e = atf::launch_decode(p, d, static_cast<hipStream_t>(hip_stream));
    if (e != hipSuccess) return fail(ATF_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return ATF_OK;
}

}  // namespace

extern "C" {

int atf_decode(const void* q, const void* k_cache, const void* v_cache, void* o, float* lse,
               int32_t batch, int64_t n_k, int64_t q_pos, int32_t h_q, int32_t h_kv,
               int64_t cache_tokens, const atf_window* w, float softmax_scale, void* workspace,
               size_t workspace_bytes, void* hip_stream) {
    return decode_impl("decode", q, k_cache, v_cache, o, lse, batch, n_k, q_pos, nullptr, nullptr,
                       h_q, h_kv, cache_tokens, w, softmax_scale, workspace, workspace_bytes,
                       hip_stream);
}

int atf_decode_noalloc(const void* q, const void* k_cache, const void* v_cache, void* o,
                       float* lse, int32_t batch, int64_t n_k, int64_t q_pos, int32_t h_q,
                       int32_t h_kv, int64_t cache_tokens, const atf_window* w,
                       float softmax_scale, void* hip_stream) {
    static_assert(atf::kNoAllocScratchBytes == ATF_DECODE_NOALLOC_SCRATCH_BYTES,
                  "scratch size of the header and of the library differ");
    if (w == nullptr) return fail(ATF_EINVAL, "decode_noalloc: NULL window");
    const int d = w->head_dim;
    if (batch >= 1 && h_q >= 1 && h_kv >= 1 && h_q % h_kv == 0 && n_k >= 1 && n_k < kPosLimit &&
        (d == 64 || d == 128)) {
        const size_t need = uniform_layout(batch, h_q, h_kv, n_k, d).total;
        if (need > atf::kNoAllocScratchBytes)
            return fail(ATF_EWORKSPACE,
                        "decode_noalloc: these sizes need %zu bytes of partial states, above the "
                        "%zu-byte scratch array (use atf_decode with a workspace)",
                        need, atf::kNoAllocScratchBytes);
    }
    void* ws = nullptr;
    const hipError_t e = atf::noalloc_scratch(&ws);
    if (e != hipSuccess)
        return fail(ATF_EHIP, "decode_noalloc: scratch address: %s", hipGetErrorString(e));
    // every other argument is checked as atf_decode checks it
    return decode_impl("decode_noalloc", q, k_cache, v_cache, o, lse, batch, n_k, q_pos, nullptr,
                       nullptr, h_q, h_kv, cache_tokens, w, softmax_scale, ws,
                       atf::kNoAllocScratchBytes, hip_stream);
}

int atf_decode_unrotated(const void* q, const void* k_cache, const void* v_cache, void* o,
                         float* lse, int32_t batch, int64_t n_k, int64_t q_pos, int32_t h_q,
                         int32_t h_kv, int64_t cache_tokens, const atf_window* w,
                         const double* rope_inv_freq, float softmax_scale, void* workspace,
                         size_t workspace_bytes, void* hip_stream) {
    RopeArgs rope;
    rope.rotate = true;
    rope.inv_freq = rope_inv_freq;
    return decode_impl("decode_unrotated", q, k_cache, v_cache, o, lse, batch, n_k, q_pos, nullptr,
                       nullptr, h_q, h_kv, cache_tokens, w, softmax_scale, workspace,
                       workspace_bytes, hip_stream, PagedArgs(), rope);
}

int atf_decode_ragged_unrotated(const void* q, const void* k_cache, const void* v_cache, void* o,
                                float* lse, int32_t batch, const int32_t* n_k_rows,
                                const int32_t* q_pos_rows, int64_t max_n_k, int32_t h_q,
                                int32_t h_kv, int64_t cache_tokens, const atf_window* w,
                                const double* rope_inv_freq, float softmax_scale,
                                void* workspace, size_t workspace_bytes, void* hip_stream) {
    if (!n_k_rows || !q_pos_rows)
        return fail(ATF_EINVAL, "decode_ragged_unrotated: NULL row-length or row-position array");
    RopeArgs rope;
    rope.rotate = true;
    rope.inv_freq = rope_inv_freq;
    return decode_impl("decode_ragged_unrotated", q, k_cache, v_cache, o, lse, batch, max_n_k, 0,
                       n_k_rows, q_pos_rows, h_q, h_kv, cache_tokens, w, softmax_scale, workspace,
                       workspace_bytes, hip_stream, PagedArgs(), rope);
}

int atf_decode_ragged(const void* q, const void* k_cache, const void* v_cache, void* o, float* lse,
                      int32_t batch, const int32_t* n_k_rows, const int32_t* q_pos_rows,
                      int64_t max_n_k, int32_t h_q, int32_t h_kv, int64_t cache_tokens,
                      const atf_window* w, float softmax_scale, void* workspace,
                      size_t workspace_bytes, void* hip_stream) {
    if (!n_k_rows || !q_pos_rows)
        return fail(ATF_EINVAL, "decode_ragged: NULL row-length or row-position array");
    return decode_impl("decode_ragged", q, k_cache, v_cache, o, lse, batch, max_n_k, 0, n_k_rows,
                       q_pos_rows, h_q, h_kv, cache_tokens, w, softmax_scale, workspace,
                       workspace_bytes, hip_stream);
}

}  // extern "C"

namespace {
int decode_paged_impl(const char* fn, const void* q, const void* k_pages, const void* v_pages,
                      void* o, float* lse, int32_t batch, const int32_t* block_table,
                      int32_t max_pages_per_row, int32_t num_pages, int32_t page_tokens,
                      const int32_t* n_k_rows, const int32_t* q_pos_rows, int64_t max_n_k,
                      int32_t h_q, int32_t h_kv, const atf_window* w, float softmax_scale,
                      void* workspace, size_t workspace_bytes, void* hip_stream,
                      const RopeArgs& rope) {
    if (!block_table) return fail(ATF_EINVAL, "%s: NULL block table", fn);
    if (!n_k_rows || !q_pos_rows)
        return fail(ATF_EINVAL, "%s: NULL row-length or row-position array", fn);
    if (page_tokens < 32 || page_tokens % 32 != 0)
        return fail(ATF_EINVAL, "%s: page_tokens %d must be a positive multiple of 32",
                    fn, page_tokens);
    if (num_pages < 1 || max_pages_per_row < 1)
        return fail(ATF_EINVAL, "%s: need num_pages >= 1 and max_pages_per_row >= 1", fn);
    const int64_t row_cap = int64_t(max_pages_per_row) * page_tokens;
    if (max_n_k > row_cap || row_cap > kPosLimit)
        return fail(ATF_EINVAL, "%s: max_n_k %lld exceeds the %lld tokens a row's pages "
                    "hold (or that exceeds 2^31 - 1)", fn, (long long)max_n_k, (long long)row_cap);
    PagedArgs pg;
    pg.block_table = block_table;
    pg.max_pages = max_pages_per_row;
    pg.num_pages = num_pages;
    pg.page_tokens = page_tokens;
    // the contiguous-cache capacity is the rows' span; the kernel addresses pages instead
    return decode_impl(fn, q, k_pages, v_pages, o, lse, batch, max_n_k, 0, n_k_rows, q_pos_rows,
                       h_q, h_kv, row_cap, w, softmax_scale, workspace, workspace_bytes, hip_stream,
                       pg, rope);
}
}  // namespace

extern "C" {

int atf_decode_paged(const void* q, const void* k_pages, const void* v_pages, void* o, float* lse,
                     int32_t batch, const int32_t* block_table, int32_t max_pages_per_row,
                     int32_t num_pages, int32_t page_tokens, const int32_t* n_k_rows,
                     const int32_t* q_pos_rows, int64_t max_n_k, int32_t h_q, int32_t h_kv,
                     const atf_window* w, float softmax_scale, void* workspace,
                     size_t workspace_bytes, void* hip_stream) {
    return decode_paged_impl("decode_paged", q, k_pages, v_pages, o, lse, batch, block_table,
                             max_pages_per_row, num_pages, page_tokens, n_k_rows, q_pos_rows,
                             max_n_k, h_q, h_kv, w, softmax_scale, workspace, workspace_bytes,
                             hip_stream, RopeArgs());
}

int atf_decode_paged_unrotated(const void* q, const void* k_pages, const void* v_pages, void* o,
                               float* lse, int32_t batch, const int32_t* block_table,
                               int32_t max_pages_per_row, int32_t num_pages, int32_t page_tokens,
                               const int32_t* n_k_rows, const int32_t* q_pos_rows,
                               int64_t max_n_k, int32_t h_q, int32_t h_kv, const atf_window* w,
                               const double* rope_inv_freq, float softmax_scale, void* workspace,
                               size_t workspace_bytes, void* hip_stream) {
    RopeArgs rope;
    rope.rotate = true;
    rope.inv_freq = rope_inv_freq;
    return decode_paged_impl("decode_paged_unrotated", q, k_pages, v_pages, o, lse, batch,
                             block_table, max_pages_per_row, num_pages, page_tokens, n_k_rows,
                             q_pos_rows, max_n_k, h_q, h_kv, w, softmax_scale, workspace,
                             workspace_bytes, hip_stream, rope);
}

namespace {
// Shared by atf_cache_append_paged and atf_cache_append_paged_rotated (rope != nullptr:
// the keys turned to their positions on the way in).
int cache_append_paged_impl(const char* fn, const void* k_new, const void* v_new, void* k_pages,
                            void* v_pages, const int32_t* block_table, int32_t max_pages_per_row,
                            int32_t num_pages, int32_t page_tokens, int32_t batch, int64_t n_new,
                            int64_t pos0, int32_t h_kv, int32_t head_dim, void* hip_stream,
                            const atf::RotatePagedParams* rope) {
    if (head_dim != 64 && head_dim != 128)
        return fail(ATF_EUNSUPPORTED, "%s: head_dim %d not built", fn, head_dim);
    if (batch < 1 || h_kv < 1 || n_new < 0 || pos0 < 0)
        return fail(ATF_EINVAL, "%s: need batch >= 1, h_kv >= 1, n_new >= 0, pos0 >= 0", fn);
    if (page_tokens < 32 || page_tokens % 32 != 0)
        return fail(ATF_EINVAL, "%s: page_tokens %d must be a positive multiple of 32", fn,
                    page_tokens);
    if (num_pages < 1 || max_pages_per_row < 1)
        return fail(ATF_EINVAL, "%s: need num_pages >= 1 and max_pages_per_row >= 1", fn);
    const int64_t row_cap = int64_t(max_pages_per_row) * page_tokens;
    if (row_cap > kPosLimit || pos0 + n_new > row_cap)
        return fail(ATF_EINVAL, "%s: tokens %lld .. %lld do not fit the %lld tokens "
                    "of a row's pages", fn, (long long)pos0, (long long)(pos0 + n_new), (long long)row_cap);
    if (!k_new || !v_new || !k_pages || !v_pages || !block_table)
        return fail(ATF_EINVAL, "%s: NULL pointer", fn);
    if (!aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k_pages, 16) ||
        !aligned(v_pages, 16) || !aligned(block_table, 4))
        return fail(ATF_EINVAL, "%s: tensors must be 16-byte, the table 4-byte aligned", fn);
    if (n_new == 0) return ATF_OK;
    if (int64_t(batch) * n_new * h_kv > kPosLimit)
        return fail(ATF_EINVAL, "%s: too many tokens for one call", fn);
    atf::AppendPagedParams p{};
    p.k_src = static_cast<const uint16_t*>(k_new);
    p.v_src = static_cast<const uint16_t*>(v_new);
    p.k_pages = static_cast<uint16_t*>(k_pages);
    p.v_pages = static_cast<uint16_t*>(v_pages);
    p.block_table = block_table;
    p.batch = batch;
    p.n_new = static_cast<int32_t>(n_new);
    p.pos0 = static_cast<int32_t>(pos0);
    p.h_kv = h_kv;
    p.max_pages = max_pages_per_row;
    p.num_pages = num_pages;
    p.page_tokens = page_tokens;
    hipError_t e;
    if (rope != nullptr) {
        atf::RotatePagedParams rp = *rope;
        rp.a = p;
        e = atf::launch_append_paged_rotated(rp, head_dim, static_cast<hipStream_t>(hip_stream));
    } else {
        e = atf::launch_append_paged(p, head_dim, static_cast<hipStream_t>(hip_stream));
    }
    if (e != hipSuccess) return fail(ATF_EHIP, "%s: launch failed: %s", fn, hipGetErrorString(e));
    return ATF_OK;
}
}  // namespace

int atf_cache_append_paged(const void* k_new, const void* v_new, void* k_pages, void* v_pages,
                           const int32_t* block_table, int32_t max_pages_per_row,
                           int32_t num_pages, int32_t page_tokens, int32_t batch, int64_t n_new,
                           int64_t pos0, int32_t h_kv, int32_t head_dim, void* hip_stream) {
    return cache_append_paged_impl("cache_append_paged", k_new, v_new, k_pages, v_pages,
                                   block_table, max_pages_per_row, num_pages, page_tokens, batch,
                                   n_new, pos0, h_kv, head_dim, hip_stream, nullptr);
}

int atf_cache_append_paged_rotated(const void* k_new, const void* v_new, void* k_pages,
                                   void* v_pages, const int32_t* block_table,
                                   int32_t max_pages_per_row, int32_t num_pages,
                                   int32_t page_tokens, int32_t batch, int64_t n_new, int64_t pos0,
                                   int32_t h_kv, const atf_window* w, const double* rope_inv_freq,
                                   void* hip_stream) {
    const char* fn = "cache_append_paged_rotated";
    if (w == nullptr) return fail(ATF_EINVAL, "%s: NULL window", fn);
    const int d = w->head_dim;
    if (d != 64 && d != 128)
        return fail(ATF_EUNSUPPORTED, "%s: head_dim %d not built (64 or 128)", fn, d);
    atf::RotatePagedParams rp{};
    const int rc = rope_fractions(fn, w, rope_inv_freq, rp.rope_rho_hi, rp.rope_rho_lo);
    if (rc != ATF_OK) return rc;
    return cache_append_paged_impl(fn, k_new, v_new, k_pages, v_pages, block_table,
                                   max_pages_per_row, num_pages, page_tokens, batch, n_new, pos0,
                                   h_kv, d, hip_stream, &rp);
}

}  // extern "C"
