// Thin projections for factored keys (Sec. 2.3, Eq. 6-7): Y = X W for one
// projection of a layer, written head-major for the attention kernels.
//
// After a pretrained key projection is factored per KV head (W_K ~= A B) and B
// is absorbed into the query projection (W_Q' = W_Q B^T), the layer computes
// r-wide queries q' = x W_Q' and keys k' = x W_K' = x A for every token, and
// its full-width values v = x W_V. Each is a dense product of the token rows
// X [tokens, d_model] with a weight matrix whose columns are grouped by head.
// This kernel computes one such product on the bf16 matrix cores with fp32
// accumulation and stores the result straight into the [batch, head, token,
// width] layout that tk_attn_prefill and tk_cache_append read, so no separate
// transpose pass follows.
//
// The weight is passed transposed, Wt [n_heads * width, d_model] (one row per
// output column), so both operands of the product are contiguous along
// d_model, which must be a multiple of 32 (one k-tile). The tile computes C^T = Wt X^T: a lane of each accumulator
// then holds four consecutive output columns of one token, which become one
// 8-byte store into the head-major output row.
#include "tk_device.hpp"
#include "tk_internal.hpp"

namespace tk {

namespace {

constexpr int kPBK = 32;   // d_model per k-tile: 4 chunks of 8 bf16 per row
constexpr int kStages = 3; // k-tiles in LDS: the one multiplied and two in flight
constexpr int kXcdCount = 8;

// A workgroup tile of BN output columns (weight rows) x BM tokens. Its waves are
// laid out (BN / 64) x 2: each owns 64 columns x BM / 2 tokens.
template <int BN, int BM>
struct ProjTile {
    static constexpr int kWaves = (BN / 64) * 2;
    static constexpr int kThreads = 64 * kWaves;
    static constexpr int kMB = BM / 64;                         // 32-token blocks per wave
    static constexpr int kWCopies = BN * kPBK / 8 / kThreads;  // copies per lane and k-tile
    static constexpr int kXCopies = BM * kPBK / 8 / kThreads;
    static constexpr int kCopies = kWCopies + kXCopies;        // a lane's copies in flight per k-tile
    static_assert(kWCopies * kThreads * 8 == BN * kPBK && kXCopies * kThreads * 8 == BM * kPBK, "tiling");
    uint16_t w[kStages][BN * kPBK];  // weight rows of the tile (swizzled 16-byte chunks)
    uint16_t x[kStages][BM * kPBK];  // token rows of the tile (same swizzle)
};

// Chunk kc (0..3) of tile row r sits in slot 4 r + (kc ^ ((r / 4) % 4)). Rows are
// 64 bytes, so four rows share one 256-byte line of the 64 LDS banks; the
// rotation gives the same chunk of the rows r, r + 4, r + 8, r + 12 four
// different 16-byte bank groups, so the 16 consecutive rows one quarter-wave
// reads cover all 64 banks once. The map is its own inverse: slot 4 r + q
// holds chunk q ^ ((r / 4) % 4).
__device__ __forceinline__ int sw(int r, int kc) { return r * kPBK + ((kc ^ ((r >> 2) & 3)) << 3); }

template <int N>
__device__ __forceinline__ void wait_copies(bool next_in_flight) {
    if (next_in_flight)
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
    else
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

// Each wave multiplies a 64-column x BM / 2-token block. Tiles come from HBM by
// global->LDS copies (no staging registers), issued two k-tiles ahead into a
// three-stage ring. The 256 x 256 tiles run 16x16x32 products in a ping-pong
// between the two waves of each SIMD; the smaller ones run 32x32x16 products,
// each wave reading the next 16-wide k-step's operands during the current one's
// products.
template <int BN>
constexpr int proj_threads() { return 64 * (BN / 64) * 2; }

template <int BN, int BM>
__global__ __launch_bounds__(proj_threads<BN>(), 1) void project_kernel(const ProjectParams p) {
    using T = ProjTile<BN, BM>;
    constexpr int kPThreads = T::kThreads, kWCopies = T::kWCopies, kXCopies = T::kXCopies;
    constexpr int kPBN = BN, kPBM = BM;
    __shared__ T sm;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wn = wave >> 1, wm = wave & 1;  // (BN / 64) x 2 waves over the tile's columns x tokens
    // XCD-aware order: workgroups are dealt to the 8 XCDs round-robin; each XCD
    // takes a contiguous range of tiles, column tiles fastest, so the column
    // tiles of one token tile run on one XCD and share its rows through its L2
    const int per_xcd = (p.tiles + kXcdCount - 1) / kXcdCount;
    const int logical = (int)(blockIdx.x % kXcdCount) * per_xcd + (int)(blockIdx.x / kXcdCount);
    if (logical >= p.tiles) return;
    const int n_tiles = (p.N + kPBN - 1) / kPBN;
    const int n_base = (logical % n_tiles) * kPBN, m_base = (logical / n_tiles) * kPBM;

    // Copy i of this lane fills LDS slot i * 256 + tid of the tile: row slot / 4,
    // chunk (slot % 4) ^ ((row / 4) % 4) of that row in the matrix. Rows past the
    // matrix re-read its last row (finite values whose outputs are not stored).
    const int wlast = (p.N - n_base < kPBN ? p.N - n_base : kPBN) - 1;
    const int xlast = (p.M - m_base < kPBM ? p.M - m_base : kPBM) - 1;
    uint32_t woff[kWCopies], xoff[kXCopies];
#pragma unroll
    for (int i = 0; i < kWCopies; ++i) {
        const int slot = i * kPThreads + tid, r = slot >> 2, kc = (slot & 3) ^ ((r >> 2) & 3);
        woff[i] = (uint32_t)(((r < wlast ? r : wlast) * p.K + kc * 8) * 2);
    }
#pragma unroll
    for (int i = 0; i < kXCopies; ++i) {
        const int slot = i * kPThreads + tid, r = slot >> 2, kc = (slot & 3) ^ ((r >> 2) & 3);
        xoff[i] = (uint32_t)(((r < xlast ? r : xlast) * p.K + kc * 8) * 2);
    }
    const char* wg = (const char*)((const uint16_t*)p.wt + (size_t)n_base * p.K);
    const char* xg = (const char*)((const uint16_t*)p.x + (size_t)m_base * p.K);
    auto issue = [&](int kt, int stage) {
        const char* wk = wg + (size_t)kt * kPBK * 2;
        const char* xk = xg + (size_t)kt * kPBK * 2;
#pragma unroll
        for (int i = 0; i < kWCopies; ++i) copy16_to_lds(wk, woff[i], sm.w[stage] + (i * kPThreads + wave * 64) * 8);
#pragma unroll
        for (int i = 0; i < kXCopies; ++i) copy16_to_lds(xk, xoff[i], sm.x[stage] + (i * kPThreads + wave * 64) * 8);
    };

    if constexpr (BM == 256) {
        // ---- 256 x 256 tiles: ping-pong over the two waves of each SIMD ----
        // The eight waves form two groups of four, one wave of each on every SIMD;
        // the second group runs one barrier behind the first. A wave reads a whole
        // k-tile's operands while the other wave of its SIMD runs its products, then
        // runs its own products (32 of 16x16x32) while the other reads: the two
        // phases alternate at every barrier. Each lane's 16-byte operand read is row
        // r16 of a 16-row block at chunk q4, the whole 32-wide k-tile over the four
        // lane groups, and an accumulator lane ends with four consecutive output
        // columns of one token. Both groups pass 2 nk + 2 barriers: the late group's
        // extra one comes first, the early group's last.
        constexpr int kNB = BM / 32;
        const int r16 = lane & 15, q4 = lane >> 4;
        f32x4 acc[4][kNB];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < kNB; ++j)
#pragma unroll
                for (int v = 0; v < 4; ++v) acc[i][j][v] = 0.f;
        const int nk = p.K / kPBK;
        issue(0, 0);
        if (nk > 1) issue(1, 1);
        wait_copies<T::kCopies>(nk > 1);
        __syncthreads();
        const bool late = wave >= 4;
        if (late) {
            __builtin_amdgcn_sched_barrier(0);
            __syncthreads();
            __builtin_amdgcn_sched_barrier(0);
        }
        bf16x8 a[4], b[kNB];
        int stage = 0;
        for (int kt = 0; kt < nk; ++kt) {
            // the stage k-tile kt + 2 goes to held k-tile kt - 1, which both groups
            // have read before the barrier that opened this wave's read phase
            const bool ahead = kt + 2 < nk;
            if (ahead) issue(kt + 2, stage == 0 ? 2 : stage - 1);
            const uint16_t* ws = sm.w[stage];
            const uint16_t* xs = sm.x[stage];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = *(const bf16x8*)(ws + sw(wn * 64 + i * 16 + r16, q4));
#pragma unroll
            for (int j = 0; j < kNB; ++j) b[j] = *(const bf16x8*)(xs + sw(wm * (BM / 2) + j * 16 + r16, q4));
            wait_copies<T::kCopies>(ahead);  // k-tile kt + 1 has landed before the next barrier
            // the schedule barriers keep the reads and products in their phases
            __builtin_amdgcn_sched_barrier(0);
            __syncthreads();
            __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < kNB; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
            __builtin_amdgcn_sched_barrier(0);
            __syncthreads();
            __builtin_amdgcn_sched_barrier(0);
            stage = stage == kStages - 1 ? 0 : stage + 1;
        }
        if (!late) {
            __builtin_amdgcn_sched_barrier(0);
            __syncthreads();
            __builtin_amdgcn_sched_barrier(0);
        }
#pragma unroll
        for (int j = 0; j < kNB; ++j) {
            const int m = m_base + wm * (BM / 2) + j * 16 + r16;
            if (m >= p.M) continue;
            const int bb = m / p.S, s = m - bb * p.S;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int n = n_base + wn * 64 + i * 16 + 4 * q4;
                if (n >= p.N) continue;
                const int h = n / p.width, w = n - h * p.width;
                uint2 v;
                v.x = pack_bf16(acc[i][j][0], acc[i][j][1]);
                v.y = pack_bf16(acc[i][j][2], acc[i][j][3]);
                *(uint2*)((uint16_t*)p.y + (((size_t)bb * p.heads + h) * p.S + s) * p.width + w) = v;
            }
        }
    } else {
        // ---- smaller tiles: 32x32x16 products, software-pipelined over k-steps ----
        const int col = lane & 31, half = lane >> 5;
        f32x16 acc[2][T::kMB];
#pragma unroll
        for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < T::kMB; ++j)
#pragma unroll
                for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

        const int nk = p.K / kPBK;
        // operand reads of k-step ks of the k-tile in `st`, and the products of one k-step
        auto read_ops = [&](int st, int ks, bf16x8 (&a)[2], bf16x8 (&b)[T::kMB]) {
            const uint16_t* ws = sm.w[st];
            const uint16_t* xs = sm.x[st];
            const int kc = 2 * ks + half;
#pragma unroll
            for (int i = 0; i < 2; ++i) a[i] = *(const bf16x8*)(ws + sw(wn * 64 + i * 32 + col, kc));
#pragma unroll
            for (int j = 0; j < T::kMB; ++j) b[j] = *(const bf16x8*)(xs + sw(wm * (BM / 2) + j * 32 + col, kc));
        };
        auto products = [&](const bf16x8 (&a)[2], const bf16x8 (&b)[T::kMB]) {
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < T::kMB; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[i], b[j], acc[i][j], 0, 0, 0);
        };
        issue(0, 0);
        if (nk > 1) issue(1, 1);
        wait_copies<T::kCopies>(nk > 1);  // this lane's copies of k-tile 0 have landed
        __syncthreads();      // ... and everyone's
        static_assert(kPBK == 32, "the pipeline below takes two 16-wide k-steps per k-tile");
        // Software pipeline over the k-steps: the operands of the next k-step are
        // read while the current one's products run, and the barrier that publishes
        // k-tile kt + 1 sits between the two k-steps of k-tile kt, so that its first
        // operand reads overlap the second k-step's products.
        bf16x8 a0[2], b0[T::kMB], a1[2], b1[T::kMB];
        read_ops(0, 0, a0, b0);
        int stage = 0;
        for (int kt = 0; kt + 1 < nk; ++kt) {
            // the stage k-tile kt + 2 goes to was last read before the barrier that
            // ended iteration kt - 1
            const bool ahead = kt + 2 < nk;
            if (ahead) issue(kt + 2, stage == 0 ? 2 : stage - 1);
            read_ops(stage, 1, a1, b1);
            products(a0, b0);
            const int next = stage == kStages - 1 ? 0 : stage + 1;
            wait_copies<T::kCopies>(ahead);  // k-tile kt + 1 has landed (kt + 2 may still fly)
            __syncthreads();
            read_ops(next, 0, a0, b0);
            products(a1, b1);
            stage = next;
        }
        // the last k-tile
        read_ops(stage, 1, a1, b1);
        products(a0, b0);
        products(a1, b1);

        // ---- epilogue: lane (col, half) of block (i, j) holds output columns
        // n0 + 8 g + 4 half + 0..3 (g = 0..3) of token m0 + col, rounded to bf16 and
        // stored as 8 bytes into Y[b, h, s, w .. w + 3]
#pragma unroll
        for (int j = 0; j < T::kMB; ++j) {
            const int m = m_base + wm * (BM / 2) + j * 32 + col;
            if (m >= p.M) continue;
            const int bb = m / p.S, s = m - bb * p.S;
#pragma unroll
            for (int i = 0; i < 2; ++i) {
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const int n = n_base + wn * 64 + i * 32 + 8 * g + 4 * half;
                    if (n >= p.N) continue;
                    const int h = n / p.width, w = n - h * p.width;
                    uint2 v;
                    v.x = pack_bf16(acc[i][j][4 * g], acc[i][j][4 * g + 1]);
                    v.y = pack_bf16(acc[i][j][4 * g + 2], acc[i][j][4 * g + 3]);
                    *(uint2*)((uint16_t*)p.y + (((size_t)bb * p.heads + h) * p.S + s) * p.width + w) = v;
                }
            }
        }
    }
}

}  // namespace

// Tile shape of a call, the largest that still gives every CU a workgroup:
// 256 x 256 (8 waves of 64 columns x 128 tokens, one workgroup per CU); else
// 256 columns x 128 tokens (8 waves of 64 x 64), which serves the narrow
// thin-key projection (a few KV heads of r columns) over long inputs with the
// token rows read once; else 128 x 128 (4 waves, two workgroups per CU), so that
// short sequences still spread over the part.
enum class ProjShape { k256x256, k256x128, k128x128 };

static long tiles_of(long M, long N, long BN, long BM) { return ((M + BM - 1) / BM) * ((N + BN - 1) / BN); }

static ProjShape shape_of(long M, long N) {
    if (tiles_of(M, N, 256, 256) >= 256) return ProjShape::k256x256;
    if (tiles_of(M, N, 256, 128) >= 256) return ProjShape::k256x128;
    return ProjShape::k128x128;
}

long project_tiles(long M, long N) {
    switch (shape_of(M, N)) {
        case ProjShape::k256x256: return tiles_of(M, N, 256, 256);
        case ProjShape::k256x128: return tiles_of(M, N, 256, 128);
        default: return tiles_of(M, N, 128, 128);
    }
}

tk_status launch_project(const ProjectParams& p, hipStream_t st) {
    const long launched = ((long)p.tiles + kXcdCount - 1) / kXcdCount * kXcdCount;
    const dim3 grid((unsigned)launched);
    switch (shape_of(p.M, p.N)) {
        case ProjShape::k256x256:
            hipLaunchKernelGGL((project_kernel<256, 256>), grid, dim3(ProjTile<256, 256>::kThreads), 0, st, p);
            break;
        case ProjShape::k256x128:
            hipLaunchKernelGGL((project_kernel<256, 128>), grid, dim3(ProjTile<256, 128>::kThreads), 0, st, p);
            break;
        default:
            hipLaunchKernelGGL((project_kernel<128, 128>), grid, dim3(ProjTile<128, 128>::kThreads), 0, st, p);
    }
    return hipGetLastError() == hipSuccess ? TK_OK : TK_ERR_HIP;
}

}  // namespace tk
