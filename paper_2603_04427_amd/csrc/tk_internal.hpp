// Internal interface between the C-ABI layer (api.cpp) and the kernel launchers.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "tk_attn.h"

namespace tk {

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Key formats of the cache: bf16 rows, OCP E4M3 codes, or 4-bit integer codes
// (excess-8 nibbles, two per byte, low nibble first); the quantised formats
// carry one fp32 scale per (token, KV head).
enum KeyFormat : int { kKeyBF16 = 0, kKeyE4M3 = 1, kKeyInt4 = 2 };

// Decode: one 256-thread workgroup per (split, KV head x head group, sequence).
struct DecodeParams {
    const uint16_t* q;          // [B, Hq, R] bf16
    const uint8_t* k;           // key rows: bf16 (2R bytes), E4M3 codes (R bytes) or 4-bit codes (R/2 bytes)
    const float* k_scale;       // per key row (fp8 only)
    const uint16_t* v;          // value rows, DV bf16
    const int32_t* ctx_lens;    // [B]
    const int32_t* block_table; // [B, mb] or null
    float* ws;                  // partials [B, Hq, n_split, DV + 2]
    unsigned* counters;         // [B, Hq] arrival counters (first B * Hq / HG used), zero between calls
    uint16_t* o;                // [B, Hq, DV] bf16
    int B, Hq, Hkv, G, max_ctx;
    int bs_log2, mb, num_blocks;
    int n_split;                // splits of each (sequence, head group): split s takes rounds s, s + n_split, ...
    float qscale;               // softmax scale * log2(e)
};

struct DecodePlan {
    int heads_per_group;  // query heads one workgroup serves (divides G, <= 8)
    int n_split;
    int split_len;  // tokens per split, a multiple of 512 (planning: n_split = ceil(max_ctx / split_len))
    size_t counter_bytes;  // leading counter region of the workspace (256-byte multiple)
    size_t ws_bytes;
};

// Pure function of the shapes (no device query).
DecodePlan plan_decode(int B, int Hq, int Hkv, int max_ctx, int DV);

tk_status launch_decode(const DecodeParams& p, int R, int DV, int HG, int key_format, bool paged,
                        hipStream_t stream);

// The library's own decode scratch, for callers that cannot allocate: one fixed
// device array per GPU (kDecodeScratchBytes), its counter region zeroed once.
// Every split plan fits: a split context needs fewer than 512 (sequence, head
// group, split) triples of at most 8 heads, 4096 partial rows of DV + 2 floats.
constexpr size_t kDecodeScratchBytes = size_t(4) << 20;
// Device address of the current device's copy (looked up and cleared on the
// first call on that device, on `stream`); TK_ERR_HIP if that fails.
tk_status decode_scratch(hipStream_t stream, void** ptr);

// Cache append: grid-stride over 16-byte row slices of the new tokens.
struct AppendParams {
    const uint16_t* kn;         // [B, Hkv, T, R] bf16 new key rows
    const uint16_t* vn;         // [B, Hkv, T, DV] bf16 new value rows
    const int32_t* pos;         // [B] first position written
    uint8_t* kc;                // key cache rows: bf16 (2R bytes), E4M3 codes (R bytes) or 4-bit codes (R/2)
    float* ks;                  // per key row scale (quantised keys only)
    uint16_t* vc;               // value cache rows
    const int32_t* table;       // [B, mb] or null
    int B, Hkv, T;
    long capacity;              // positions per sequence: max_ctx, or block_size * mb when paged
    int bs_log2, mb, num_blocks;
};

tk_status launch_append(const AppendParams& p, int R, int DV, int key_format, bool paged, hipStream_t stream);

struct PrefillParams {
    const void* q;   // [B, Hq, Sq, R]
    const void* k;   // [B, Hkv, Sk, R]
    const void* v;   // [B, Hkv, Sk, DV]
    void* o;         // [B, Hq, Sq, DV]
    float* lse;      // [B, Hq, Sq] natural-log log-sum-exp of the scaled scores, or null (bf16 only)
    int B, Hq, Hkv, G, Sq, Sk;
    int causal;
    float qscale;    // softmax scale * log2(e)
};

// Prefill backward (bf16): dQ with D = rowsum(dO * O), then dK and dV.
struct PrefillBwdParams {
    const void* q;      // [B, Hq, Sq, R]
    const void* k;      // [B, Hkv, Sk, R]
    const void* v;      // [B, Hkv, Sk, DV]
    const void* o;      // [B, Hq, Sq, DV]   forward output
    const void* dout;   // [B, Hq, Sq, DV]   gradient of the output
    const float* lse;   // [B, Hq, Sq]       forward log-sum-exp (natural log)
    void* dq;           // [B, Hq, Sq, R]
    void* dk;           // [B, Hkv, Sk, R]
    void* dv;           // [B, Hkv, Sk, DV]
    float* delta;       // [B, Hq, Sq] workspace: D of each row
    float* lse2;        // [B, Hq, Sq] workspace: the rows' log-sum-exp in log2 units
    int B, Hq, Hkv, G, Sq, Sk;
    int causal;
    float scale;        // softmax scale
    float qscale;       // scale * log2(e)
};

tk_status launch_prefill_backward(const PrefillBwdParams& p, int R, int DV, hipStream_t stream);

// Thin projection: Y[b, h, s, w] = sum_k X[b, s, k] Wt[h * width + w, k] (bf16
// in, fp32 accumulation, bf16 out).
struct ProjectParams {
    const void* x;   // [M = batch * S, K] bf16 token rows
    const void* wt;  // [N = heads * width, K] bf16, the weight's columns as rows
    void* y;         // [batch, heads, S, width] bf16
    int M, N, K, S, heads, width;
    int tiles;       // 128 x 128 output tiles
};

long project_tiles(long M, long N);
tk_status launch_project(const ProjectParams& p, hipStream_t stream);

tk_status launch_prefill_bf16(const PrefillParams& p, int R, int DV, hipStream_t stream);
tk_status launch_prefill_f32(const PrefillParams& p, int R, int DV, hipStream_t stream);

}  // namespace tk
