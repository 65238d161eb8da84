// C-ABI entry points of libtkattn: argument validation (pure host code, no HIP
// call until it passes), decode planning and kernel dispatch.
#include <math.h>
#include <stddef.h>
#include <stdint.h>

#include "tk_attn.h"
#include "tk_internal.hpp"

namespace {

bool supported_r(int r) { return r == 16 || r == 32 || r == 64 || r == 128; }
bool supported_dv(int dv) { return dv == 64 || dv == 128; }
bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

float resolve_scale(float scale, int r) { return (scale > 0.f && !isnan(scale)) ? scale : 1.0f / sqrtf((float)r); }

int log2_exact(int x) {
    int l = 0;
    while ((1 << l) < x) ++l;
    return (1 << l) == x ? l : -1;
}

constexpr long kMaxGrid = 65535;

int key_format(tk_dtype k) { return k == TK_FP8_E4M3 ? 1 : (k == TK_INT4 ? 2 : 0); }

tk_status prefill_impl(const void* Q, const void* K, const void* V, void* O, float* lse, int batch, int H_q,
                       int H_kv, int seq_q, int seq_k, int r, int d_v, int causal, float scale, tk_dtype dtype,
                       hipStream_t stream) {
    if (batch < 0 || H_q <= 0 || H_kv <= 0 || seq_q < 0 || seq_k < 0 || r <= 0 || d_v <= 0)
        return TK_ERR_INVALID_ARG;
    if (H_q % H_kv != 0) return TK_ERR_INVALID_ARG;
    if (dtype != TK_F32 && dtype != TK_BF16) return dtype == TK_FP8_E4M3 ? TK_ERR_UNSUPPORTED : TK_ERR_INVALID_ARG;
    if (causal && seq_q > seq_k) return TK_ERR_INVALID_ARG;
    if (batch == 0 || seq_q == 0) return TK_OK;
    if (seq_k == 0) return TK_ERR_INVALID_ARG;
    if (!Q || !K || !V || !O) return TK_ERR_INVALID_ARG;
    if (!aligned16(Q) || !aligned16(K) || !aligned16(V) || !aligned16(O)) return TK_ERR_INVALID_ARG;
    if (lse && ((uintptr_t)lse & 3u) != 0) return TK_ERR_INVALID_ARG;
    if (!supported_r(r) || !supported_dv(d_v)) return TK_ERR_UNSUPPORTED;
    const int G = H_q / H_kv;
    const int hpw = (G % 4 == 0) ? 4 : (G % 2 == 0 ? 2 : 1);
    const long bm = 32L * (4 / hpw);
    if ((seq_q + bm - 1) / bm > 0x7fffffffL || (long)H_kv * (G / hpw) > kMaxGrid || batch > kMaxGrid)
        return TK_ERR_UNSUPPORTED;

    tk::PrefillParams p{};
    p.q = Q;
    p.k = K;
    p.v = V;
    p.o = O;
    p.lse = lse;
    p.B = batch;
    p.Hq = H_q;
    p.Hkv = H_kv;
    p.G = G;
    p.Sq = seq_q;
    p.Sk = seq_k;
    p.causal = causal ? 1 : 0;
    p.qscale = resolve_scale(scale, r) * tk::kLog2e;
    return dtype == TK_BF16 ? tk::launch_prefill_bf16(p, r, d_v, stream) : tk::launch_prefill_f32(p, r, d_v, stream);
}

// Decode with a caller's workspace, or (use_scratch) with the library's fixed
// scratch, which then needs only the bytes the plan touches: the counters, and
// the partials when the context is split.
tk_status decode_impl(const void* Q, const void* K_cache, const void* V_cache, void* O, int batch, int H_q,
                      int H_kv, const int32_t* ctx_lens, int max_ctx, int r, int d_v, float scale, tk_dtype k_dtype,
                      const float* k_scale, const int32_t* block_table, int block_size, int max_blocks_per_seq,
                      int num_blocks, void* workspace, size_t workspace_bytes, bool use_scratch,
                      hipStream_t stream) {
    if (batch < 0 || H_q <= 0 || H_kv <= 0 || max_ctx < 0 || r <= 0 || d_v <= 0) return TK_ERR_INVALID_ARG;
    if (H_q % H_kv != 0) return TK_ERR_INVALID_ARG;
    if (k_dtype != TK_BF16 && k_dtype != TK_FP8_E4M3 && k_dtype != TK_INT4)
        return k_dtype == TK_F32 ? TK_ERR_UNSUPPORTED : TK_ERR_INVALID_ARG;
    const bool quantised = k_dtype != TK_BF16;
    if (quantised != (k_scale != nullptr)) return TK_ERR_INVALID_ARG;  // scales iff quantised keys
    const bool paged = block_table != nullptr;
    int bs_log2 = 0;
    if (paged) {
        if (block_size <= 0 || max_blocks_per_seq <= 0 || num_blocks <= 0) return TK_ERR_INVALID_ARG;
        if ((long)block_size * max_blocks_per_seq < max_ctx) return TK_ERR_INVALID_ARG;
        bs_log2 = log2_exact(block_size);
        if (bs_log2 < 0 || block_size < 64) return TK_ERR_UNSUPPORTED;
    } else if (block_size != 0 || max_blocks_per_seq != 0 || num_blocks != 0) {
        return TK_ERR_INVALID_ARG;  // layout arguments without a table
    }
    if (batch == 0) return TK_OK;
    if (!Q || !K_cache || !V_cache || !O || !ctx_lens) return TK_ERR_INVALID_ARG;
    if (!aligned16(Q) || !aligned16(K_cache) || !aligned16(V_cache) || !aligned16(O)) return TK_ERR_INVALID_ARG;
    if (!supported_r(r) || !supported_dv(d_v)) return TK_ERR_UNSUPPORTED;
    if (batch > kMaxGrid) return TK_ERR_UNSUPPORTED;

    const tk::DecodePlan pl = tk::plan_decode(batch, H_q, H_kv, max_ctx, d_v);
    if ((long)H_kv * (H_q / H_kv / pl.heads_per_group) > kMaxGrid || pl.n_split > 0x7fffffff)
        return TK_ERR_UNSUPPORTED;
    // wide keys leave no registers for 8 heads per workgroup: use groups of 4
    const int hg = (r >= 64 && pl.heads_per_group > 4) ? 4 : pl.heads_per_group;
    // a split context needs one arrival counter per (sequence, head group)
    if (pl.n_split > 1 && (size_t)batch * H_kv * (H_q / H_kv / hg) * sizeof(unsigned) > pl.counter_bytes)
        return TK_ERR_UNSUPPORTED;
    if (use_scratch) {
        const size_t need = pl.n_split > 1 ? pl.ws_bytes : pl.counter_bytes;
        if (need > tk::kDecodeScratchBytes) return TK_ERR_WORKSPACE;
        const tk_status st = tk::decode_scratch(stream, &workspace);  // first HIP call of this path
        if (st != TK_OK) return st;
    } else if (!workspace || workspace_bytes < pl.ws_bytes || ((uintptr_t)workspace & 255u)) {
        return TK_ERR_WORKSPACE;
    }

    tk::DecodeParams p{};
    p.q = (const uint16_t*)Q;
    p.k = (const uint8_t*)K_cache;
    p.k_scale = k_scale;
    p.v = (const uint16_t*)V_cache;
    p.ctx_lens = ctx_lens;
    p.block_table = block_table;
    p.counters = (unsigned*)workspace;
    p.ws = (float*)((char*)workspace + pl.counter_bytes);
    p.o = (uint16_t*)O;
    p.B = batch;
    p.Hq = H_q;
    p.Hkv = H_kv;
    p.G = H_q / H_kv;
    p.max_ctx = max_ctx;
    p.bs_log2 = bs_log2;
    p.mb = paged ? max_blocks_per_seq : 0;
    p.num_blocks = paged ? num_blocks : 0;
    p.n_split = pl.n_split;
    p.qscale = resolve_scale(scale, r) * tk::kLog2e;
    return tk::launch_decode(p, r, d_v, hg, key_format(k_dtype), paged, stream);
}

}  // namespace

extern "C" {

const char* tk_status_str(tk_status s) {
    switch (s) {
        case TK_OK: return "ok";
        case TK_ERR_INVALID_ARG: return "invalid argument";
        case TK_ERR_UNSUPPORTED: return "unsupported configuration";
        case TK_ERR_WORKSPACE: return "workspace missing or too small";
        case TK_ERR_HIP: return "HIP runtime error";
        default: return "unknown status";
    }
}

int tk_version(void) { return 100; }  // 0.1.0

tk_status tk_attn_prefill(const void* Q, const void* K, const void* V, void* O, int batch, int H_q, int H_kv,
                          int seq_q, int seq_k, int r, int d_v, int causal, float scale, tk_dtype dtype,
                          hipStream_t stream) {
    return prefill_impl(Q, K, V, O, nullptr, batch, H_q, H_kv, seq_q, seq_k, r, d_v, causal, scale, dtype, stream);
}

tk_status tk_attn_prefill_lse(const void* Q, const void* K, const void* V, void* O, float* lse, int batch, int H_q,
                              int H_kv, int seq_q, int seq_k, int r, int d_v, int causal, float scale,
                              hipStream_t stream) {
    if (!lse && batch > 0 && seq_q > 0) return TK_ERR_INVALID_ARG;
    return prefill_impl(Q, K, V, O, lse, batch, H_q, H_kv, seq_q, seq_k, r, d_v, causal, scale, TK_BF16, stream);
}

size_t tk_attn_prefill_backward_workspace_bytes(int batch, int H_q, int seq_q) {
    if (batch < 0 || H_q <= 0 || seq_q < 0) return 0;
    size_t rows = (size_t)batch * (size_t)H_q * (size_t)seq_q;
    rows = rows > 0 ? rows : 1;
    return (2 * rows * sizeof(float) + 255) / 256 * 256;
}

tk_status tk_attn_prefill_backward(const void* Q, const void* K, const void* V, const void* O, const void* dO,
                                   const float* lse, void* dQ, void* dK, void* dV, int batch, int H_q, int H_kv,
                                   int seq_q, int seq_k, int r, int d_v, int causal, float scale, void* workspace,
                                   size_t workspace_bytes, hipStream_t stream) {
    if (batch < 0 || H_q <= 0 || H_kv <= 0 || seq_q < 0 || seq_k < 0 || r <= 0 || d_v <= 0)
        return TK_ERR_INVALID_ARG;
    if (H_q % H_kv != 0) return TK_ERR_INVALID_ARG;
    if (causal && seq_q > seq_k) return TK_ERR_INVALID_ARG;
    if (seq_k == 0 && seq_q > 0) return TK_ERR_INVALID_ARG;
    if (batch == 0 || seq_k == 0) return TK_OK;
    if (!K || !V || !dK || !dV) return TK_ERR_INVALID_ARG;
    if (seq_q > 0 && (!Q || !O || !dO || !lse || !dQ)) return TK_ERR_INVALID_ARG;
    if (!aligned16(K) || !aligned16(V) || !aligned16(dK) || !aligned16(dV)) return TK_ERR_INVALID_ARG;
    if (seq_q > 0 && (!aligned16(Q) || !aligned16(O) || !aligned16(dO) || !aligned16(dQ) ||
                      ((uintptr_t)lse & 3u) != 0))
        return TK_ERR_INVALID_ARG;
    if (!workspace || ((uintptr_t)workspace & 3u) != 0 ||
        workspace_bytes < tk_attn_prefill_backward_workspace_bytes(batch, H_q, seq_q))
        return TK_ERR_WORKSPACE;
    if ((r != 32 && r != 64 && r != 128) || !supported_dv(d_v)) return TK_ERR_UNSUPPORTED;
    const int G = H_q / H_kv;
    if ((long)batch * H_q * (long)(seq_q > seq_k ? seq_q : seq_k) > 0x7fffffffL) return TK_ERR_UNSUPPORTED;

    tk::PrefillBwdParams p{};
    p.q = Q;
    p.k = K;
    p.v = V;
    p.o = O;
    p.dout = dO;
    p.lse = lse;
    p.dq = dQ;
    p.dk = dK;
    p.dv = dV;
    p.delta = (float*)workspace;
    p.lse2 = p.delta + (size_t)batch * H_q * seq_q;
    p.B = batch;
    p.Hq = H_q;
    p.Hkv = H_kv;
    p.G = G;
    p.Sq = seq_q;
    p.Sk = seq_k;
    p.causal = causal ? 1 : 0;
    p.scale = resolve_scale(scale, r);
    p.qscale = p.scale * tk::kLog2e;
    return tk::launch_prefill_backward(p, r, d_v, stream);
}

size_t tk_attn_decode_workspace_bytes(int batch, int H_q, int H_kv, int max_ctx, int d_v) {
    if (batch <= 0 || H_q <= 0 || H_kv <= 0 || H_q % H_kv != 0 || max_ctx < 0 || d_v <= 0) return 0;
    return tk::plan_decode(batch, H_q, H_kv, max_ctx, d_v).ws_bytes;
}

tk_status tk_attn_decode(const void* Q, const void* K_cache, const void* V_cache, void* O, int batch, int H_q,
                         int H_kv, const int32_t* ctx_lens, int max_ctx, int r, int d_v, float scale,
                         tk_dtype k_dtype, const float* k_scale, const int32_t* block_table, int block_size,
                         int max_blocks_per_seq, int num_blocks, void* workspace, size_t workspace_bytes,
                         hipStream_t stream) {
    return decode_impl(Q, K_cache, V_cache, O, batch, H_q, H_kv, ctx_lens, max_ctx, r, d_v, scale, k_dtype, k_scale,
                       block_table, block_size, max_blocks_per_seq, num_blocks, workspace, workspace_bytes, false,
                       stream);
}

tk_status tk_attn_decode_noalloc(const void* Q, const void* K_cache, const void* V_cache, void* O, int batch,
                                 int H_q, int H_kv, const int32_t* ctx_lens, int max_ctx, int r, int d_v,
                                 float scale, tk_dtype k_dtype, const float* k_scale, const int32_t* block_table,
                                 int block_size, int max_blocks_per_seq, int num_blocks, hipStream_t stream) {
    return decode_impl(Q, K_cache, V_cache, O, batch, H_q, H_kv, ctx_lens, max_ctx, r, d_v, scale, k_dtype, k_scale,
                       block_table, block_size, max_blocks_per_seq, num_blocks, nullptr, 0, true, stream);
}

tk_status tk_project_heads(const void* X, const void* Wt, void* Y, int batch, int seq, int d_model, int n_heads,
                           int width, hipStream_t stream) {
    if (batch < 0 || seq < 0 || d_model <= 0 || n_heads <= 0 || width <= 0) return TK_ERR_INVALID_ARG;
    if (batch == 0 || seq == 0) return TK_OK;
    if (!X || !Wt || !Y) return TK_ERR_INVALID_ARG;
    if (!aligned16(X) || !aligned16(Wt) || !aligned16(Y)) return TK_ERR_INVALID_ARG;
    if (d_model % 32 != 0 || width % 4 != 0) return TK_ERR_UNSUPPORTED;
    if (d_model > (1 << 22)) return TK_ERR_UNSUPPORTED;  // 32-bit copy offsets within a 256-row tile
    const long M = (long)batch * seq, N = (long)n_heads * width;
    if (M > 0x7fffffffL || N > 0x7fffffffL || tk::project_tiles(M, N) > 0x7fffffffL - 8) return TK_ERR_UNSUPPORTED;
    tk::ProjectParams p{};
    p.x = X;
    p.wt = Wt;
    p.y = Y;
    p.M = (int)M;
    p.N = (int)N;
    p.K = d_model;
    p.S = seq;
    p.heads = n_heads;
    p.width = width;
    p.tiles = (int)tk::project_tiles(M, N);
    return tk::launch_project(p, stream);
}

tk_status tk_cache_append(const void* K_new, const void* V_new, int batch, int H_kv, int n_new, int r, int d_v,
                          const int32_t* positions, void* K_cache, void* V_cache, int max_ctx, tk_dtype k_dtype,
                          float* k_scale, const int32_t* block_table, int block_size, int max_blocks_per_seq,
                          int num_blocks, hipStream_t stream) {
    if (batch < 0 || H_kv <= 0 || n_new < 0 || r <= 0 || d_v <= 0 || max_ctx < 0) return TK_ERR_INVALID_ARG;
    if (k_dtype != TK_BF16 && k_dtype != TK_FP8_E4M3 && k_dtype != TK_INT4)
        return k_dtype == TK_F32 ? TK_ERR_UNSUPPORTED : TK_ERR_INVALID_ARG;
    const bool quantised = k_dtype != TK_BF16;
    if (quantised != (k_scale != nullptr)) return TK_ERR_INVALID_ARG;  // scales iff quantised keys
    const bool paged = block_table != nullptr;
    int bs_log2 = 0;
    long capacity = max_ctx;
    if (paged) {
        if (block_size <= 0 || max_blocks_per_seq <= 0 || num_blocks <= 0) return TK_ERR_INVALID_ARG;
        bs_log2 = log2_exact(block_size);
        if (bs_log2 < 0) return TK_ERR_UNSUPPORTED;
        capacity = (long)block_size * max_blocks_per_seq;
    } else if (block_size != 0 || max_blocks_per_seq != 0 || num_blocks != 0) {
        return TK_ERR_INVALID_ARG;  // layout arguments without a table
    }
    if (batch == 0 || n_new == 0) return TK_OK;
    if (!K_new || !V_new || !positions || !K_cache || !V_cache) return TK_ERR_INVALID_ARG;
    if (!aligned16(K_new) || !aligned16(V_new) || !aligned16(K_cache) || !aligned16(V_cache))
        return TK_ERR_INVALID_ARG;
    if (!supported_r(r) || !supported_dv(d_v)) return TK_ERR_UNSUPPORTED;
    // 32-bit slice indices within one (sequence, KV head); at most 65535 pairs
    if ((long)n_new * (d_v > r ? d_v : r) / 8 > 0x7fffff00L || (long)batch * H_kv > kMaxGrid)
        return TK_ERR_UNSUPPORTED;

    tk::AppendParams p{};
    p.kn = (const uint16_t*)K_new;
    p.vn = (const uint16_t*)V_new;
    p.pos = positions;
    p.kc = (uint8_t*)K_cache;
    p.ks = k_scale;
    p.vc = (uint16_t*)V_cache;
    p.table = block_table;
    p.B = batch;
    p.Hkv = H_kv;
    p.T = n_new;
    p.capacity = capacity;
    p.bs_log2 = bs_log2;
    p.mb = paged ? max_blocks_per_seq : 0;
    p.num_blocks = paged ? num_blocks : 0;
    return tk::launch_append(p, r, d_v, key_format(k_dtype), paged, stream);
}

}  // extern "C"
