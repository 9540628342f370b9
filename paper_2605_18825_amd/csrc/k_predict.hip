// Multi-turn session predictor (Sec. 3.3): y = W3 relu(W2 relu(W1 h + b1) + b2) + b3
// over a batch of last-token hidden states, on the matrix cores.
//
// Layer 1 (n x d) . (d x 256) is the one dense contraction of the method:
// bf16 products (exact) summed in fp32 by v_mfma_f32_32x32x16_bf16.  A
// workgroup of 4 waves computes a 64 x 64 tile, each wave a 32 x 32 block.
// The sum over k is order-free, so A and B may share any permutation of k:
// lane l (row / column l mod 32, half l / 32) supplies, in a 64-wide k step,
// the 32 contiguous values of its half (64 bytes, four 16-byte loads), and
// MFMA m of the step takes values 8m .. 8m + 7 of both operands.  The next
// step's loads are issued before this step's four MFMAs.  Tiles are ordered
// so that the four column tiles of a row tile land on the same XCD (block
// ids go round-robin over the 8 XCDs) and read the same hidden-state rows
// through one L2.
//
// Layers 2 and 3 are fp32: v_mfma_f32_32x32x2f32 for (32 rows x 256) . (256 x
// 64) in a workgroup of 8 waves (two column halves times four k quarters,
// every load of a wave issued at once, the quarters summed in a fixed order),
// then the 64-term layer 3 by shuffles.  Layer 1's four k
// slices are added here, in slice order, before b1 and the ReLU.
#include "sae_internal.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int L1_THREADS = 256;  // 4 waves, each 64 x 64 (2 x 2 MFMA blocks of 32 x 32)
constexpr int L1_TILE = 128;       // rows and columns of a workgroup's tile
constexpr int KSTEP = 64;          // k per step
constexpr int KSPLIT = 4;          // k slices (workgroups per tile); their sums meet in layer 2
constexpr int LDS_ROW16 = 9;       // LDS row of a tile: 128 bytes of k + 16 bytes of padding
constexpr int L23_THREADS = 512;   // 8 waves: layer-2 columns 0-31 / 32-63 times k quarters
constexpr int L23_ROWS = 32;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v)
{
    bf16x8 r;
    __builtin_memcpy(&r, &v, sizeof(r));
    return r;
}

// One step (64 k) of a thread's share of the A and B tiles: rows j = 0..3.
struct Stage {
    uint4 a0, a1, a2, a3, b0, b1, b2, b3;
};

__device__ __forceinline__ void load_stage(Stage &x, const uint4 *ga0, const uint4 *ga1, const uint4 *ga2,
                                           const uint4 *ga3, const uint4 *gb0, long long bstride, int step,
                                           int nsteps)
{
    // a step past the end loads the last one (in bounds) and is zeroed, so
    // that multiplying it adds nothing
    const bool in = step < nsteps;
    const int o = (in ? step : nsteps - 1) * (KSTEP / 8);
    const uint32_t mk = in ? 0xFFFFFFFFu : 0u;  // a mask, not a select (a select of vectors
                                                // is turned into a scratch lookup)
    auto m = [mk](uint4 v) { return make_uint4(v.x & mk, v.y & mk, v.z & mk, v.w & mk); };
    x.a0 = m(ga0[o]);
    x.a1 = m(ga1[o]);
    x.a2 = m(ga2[o]);
    x.a3 = m(ga3[o]);
    x.b0 = m(gb0[o]);
    x.b1 = m(gb0[bstride + o]);
    x.b2 = m(gb0[2 * bstride + o]);
    x.b3 = m(gb0[3 * bstride + o]);
}

__device__ __forceinline__ void put_stage(const Stage &x, uint4 *la, uint4 *lb, int ls, int lstride)
{
    la[ls] = x.a0;
    la[ls + lstride] = x.a1;
    la[ls + 2 * lstride] = x.a2;
    la[ls + 3 * lstride] = x.a3;
    lb[ls] = x.b0;
    lb[ls + lstride] = x.b1;
    lb[ls + 2 * lstride] = x.b2;
    lb[ls + 3 * lstride] = x.b3;
}

// The 16 MFMAs of one step for a wave's 64 x 64 quarter (2 x 2 blocks).
__device__ __forceinline__ void mfma_step(floatx16 (&acc)[2][2], const uint4 *tla, const uint4 *tlb, int wr, int wc,
                                          int orow, int och)
{
    const uint4 *la = tla + (wr * 64 + orow) * LDS_ROW16 + och;
    const uint4 *lb = tlb + (wc * 64 + orow) * LDS_ROW16 + och;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        const bf16x8 a0 = as_bf16x8(la[m]), a1 = as_bf16x8(la[32 * LDS_ROW16 + m]);
        const bf16x8 b0 = as_bf16x8(lb[m]), b1 = as_bf16x8(lb[32 * LDS_ROW16 + m]);
        acc[0][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0][0], 0, 0, 0);
        acc[0][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b1, acc[0][1], 0, 0, 0);
        acc[1][0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1][0], 0, 0, 0);
        acc[1][1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b1, acc[1][1], 0, 0, 0);
    }
}

// One workgroup per compute unit (its LDS alone rules out three): let a
// wave use the whole register file rather than spill the pipeline stages.
__global__ void __launch_bounds__(L1_THREADS) __attribute__((amdgpu_waves_per_eu(1, 1)))
k_pred_l1(int n, int d, const uint16_t *h, const uint16_t *w1,
                                                       float *part, int row_tiles)
{
    // LDS: two stages of the A tile (128 rows) and the B tile (128 columns),
    // 64 k each, rows padded to 144 bytes so that the 32 rows one MFMA operand
    // read touches spread over the banks
    __shared__ uint4 lds[2][2][L1_TILE * LDS_ROW16];
    const int bid = blockIdx.x;
    const int xcd = bid & 7, slot = bid >> 3;
    const int ks = slot % KSPLIT;                      // k slice
    const int ct = (slot / KSPLIT) % (SAE_PRED_H1 / L1_TILE);
    const int rt = (slot / KSPLIT / (SAE_PRED_H1 / L1_TILE)) * 8 + xcd;
    if (rt >= row_tiles) return;                      // the whole workgroup
    const int tid = threadIdx.x;
    const int lane = (int)__lane_id(), wave = tid / SAE_WAVE;
    const int wr = wave >> 1, wc = wave & 1;           // this wave's 64 x 64 quarter
    const int kper = d / KSPLIT;                       // a multiple of 64
    const int kbeg = ks * kper, nsteps = kper / KSTEP;
    // global -> LDS: thread t moves 16-byte chunks of rows t / 8 + 32 j (j < 4),
    // chunk t mod 8 of each row's 128 bytes, of both tiles
    const int lr = tid >> 3, lc = tid & 7;
    const uint4 *ga0, *ga1, *ga2, *ga3;
    {
        auto arow = [&](int j) {
            int r = rt * L1_TILE + lr + 32 * j;
            r = r < n ? r : n - 1;  // rows past n repeat row n - 1 (results dropped)
            return reinterpret_cast<const uint4 *>(h + (long long)r * d + kbeg) + lc;
        };
        ga0 = arow(0);
        ga1 = arow(1);
        ga2 = arow(2);
        ga3 = arow(3);
    }
    const uint4 *gb0 = reinterpret_cast<const uint4 *>(w1 + (long long)(ct * L1_TILE + lr) * d + kbeg) + lc;
    const long long bstride = 32ll * d / 8;  // 32 rows of W1, in uint4
    const int ls = lr * LDS_ROW16 + lc, lstride = 32 * LDS_ROW16;
    floatx16 acc[2][2];
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
#pragma unroll
            for (int i = 0; i < 16; ++i) acc[bi][bj][i] = 0.0f;
    // operand reads: lane (row / column l mod 32, half l / 32) takes, in MFMA
    // m of a step, the 16 bytes at k = 32 half + 8 m of its row
    const int orow = lane & 31, och = (lane >> 5) * 4;
    // pipeline: step s is in LDS buffer s mod 2 while steps s + 1 and s + 2
    // are in flight in two register stages (the loop is unrolled by two so
    // that each stage is a fixed set of registers; a step past the end is
    // all zeros)
    Stage s0, s1;
    load_stage(s0, ga0, ga1, ga2, ga3, gb0, bstride, 0, nsteps);
    put_stage(s0, lds[0][0], lds[0][1], ls, lstride);
    load_stage(s0, ga0, ga1, ga2, ga3, gb0, bstride, 1, nsteps);
    load_stage(s1, ga0, ga1, ga2, ga3, gb0, bstride, 2, nsteps);
    __syncthreads();
    for (int st = 0; st < nsteps; st += 2) {
        mfma_step(acc, lds[0][0], lds[0][1], wr, wc, orow, och);               // step st
        put_stage(s0, lds[1][0], lds[1][1], ls, lstride);                       // step st + 1
        load_stage(s0, ga0, ga1, ga2, ga3, gb0, bstride, st + 3, nsteps);
        __syncthreads();
        mfma_step(acc, lds[1][0], lds[1][1], wr, wc, orow, och);               // step st + 1 (zeros past the end)
        put_stage(s1, lds[0][0], lds[0][1], ls, lstride);                       // step st + 2
        load_stage(s1, ga0, ga1, ga2, ga3, gb0, bstride, st + 4, nsteps);
        __syncthreads();
    }
    // partial sums of this k slice; C layout: lane l holds column l mod 32,
    // rows 8 (i / 4) + 4 (l / 32) + i mod 4 of each 32 x 32 block
    float *out = part + (long long)ks * n * SAE_PRED_H1;
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj) {
            const int col = ct * L1_TILE + wc * 64 + bj * 32 + (lane & 31);
#pragma unroll
            for (int i = 0; i < 16; ++i) {
                const int r = rt * L1_TILE + wr * 64 + bi * 32 + (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3);
                if (r < n) out[(long long)r * SAE_PRED_H1 + col] = acc[bi][bj][i];
            }
        }
}

__global__ void __launch_bounds__(L23_THREADS) __attribute__((amdgpu_waves_per_eu(1, 2)))
k_pred_l23(int n, const float *part, const float *b1, const float *w2, const float *b2, const float *w3,
           const float *b3, float *logit, uint8_t *pred)
{
    // wave w: layer-2 units 32 (w & 1) .. + 31 over k quarter w >> 1 (64 k);
    // the quarters meet in LDS and are added in quarter order
    constexpr int NQ = 4;
    __shared__ float hsum[NQ - 1][2][16][SAE_WAVE];
    __shared__ float ysum[2][L23_ROWS];
    const int lane = (int)__lane_id(), wave = threadIdx.x / SAE_WAVE;
    const int ctile = wave & 1, g = wave >> 1;
    const int r0 = blockIdx.x * L23_ROWS;
    const int row = r0 + (lane & 31);
    const int rowc = row < n ? row : n - 1;
    const int col = ctile * 32 + (lane & 31);  // layer-2 unit
    const int kb = g * (SAE_PRED_H1 / NQ) + (lane >> 5) * (SAE_PRED_H1 / NQ / 2);
    // lane half h supplies k = 64 g + 32 h + s in MFMA s, for both operands;
    // the layer-1 value is the sum of its k slices in slice order, plus b1, ReLU
    const long long slice = (long long)n * SAE_PRED_H1 / 4;  // in float4
    const float4 *pa = reinterpret_cast<const float4 *>(part + (long long)rowc * SAE_PRED_H1 + kb);
    const float4 *pb = reinterpret_cast<const float4 *>(w2 + (long long)col * SAE_PRED_H1 + kb);
    const float4 *pc = reinterpret_cast<const float4 *>(b1 + kb);
    float4 v[KSPLIT][8], b[8], c[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {  // every load of the wave in flight together
#pragma unroll
        for (int q = 0; q < KSPLIT; ++q) v[q][u] = pa[q * slice + u];
        b[u] = pb[u];
        c[u] = pc[u];
    }
    __builtin_amdgcn_sched_barrier(0);
    floatx16 acc;
#pragma unroll
    for (int i = 0; i < 16; ++i) acc[i] = 0.0f;
#pragma unroll
    for (int u = 0; u < 8; ++u) {
        float4 a = v[0][u];
#pragma unroll
        for (int q = 1; q < KSPLIT; ++q) {
            a.x = a.x + v[q][u].x;
            a.y = a.y + v[q][u].y;
            a.z = a.z + v[q][u].z;
            a.w = a.w + v[q][u].w;
        }
        a.x = a.x + c[u].x;
        a.y = a.y + c[u].y;
        a.z = a.z + c[u].z;
        a.w = a.w + c[u].w;
        a.x = a.x > 0.0f ? a.x : 0.0f;
        a.y = a.y > 0.0f ? a.y : 0.0f;
        a.z = a.z > 0.0f ? a.z : 0.0f;
        a.w = a.w > 0.0f ? a.w : 0.0f;
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.x, b[u].x, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.y, b[u].y, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.z, b[u].z, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a.w, b[u].w, acc, 0, 0, 0);
    }
    if (g > 0) {
#pragma unroll
        for (int i = 0; i < 16; ++i) hsum[g - 1][ctile][i][lane] = acc[i];
    }
    __syncthreads();
    if (g == 0) {
        // layer 2 complete (quarters in order); layer 3: this lane's column
        // weight times relu(h2) for its 16 rows, summed over the wave's 32
        // columns (lanes of one half share rows)
        const float bias = b2[col], wt = w3[col];
        float t[16];
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            float h2 = acc[i];
#pragma unroll
            for (int q = 0; q < NQ - 1; ++q) h2 = h2 + hsum[q][ctile][i][lane];
            h2 = h2 + bias;
            t[i] = wt * (h2 > 0.0f ? h2 : 0.0f);
        }
#pragma unroll
        for (int o = 1; o < 32; o <<= 1)
#pragma unroll
            for (int i = 0; i < 16; ++i) t[i] = t[i] + __shfl_xor(t[i], o);
        if ((lane & 31) == 0) {
#pragma unroll
            for (int i = 0; i < 16; ++i) ysum[ctile][(i >> 2) * 8 + (lane >> 5) * 4 + (i & 3)] = t[i];
        }
    }
    __syncthreads();
    if (threadIdx.x < L23_ROWS) {
        const int r = r0 + threadIdx.x;
        const float y = (ysum[0][threadIdx.x] + ysum[1][threadIdx.x]) + b3[0];
        if (r < n) {
            logit[r] = y;
            if (pred) pred[r] = y > 0.0f ? 1 : 0;
        }
    }
}

}  // namespace

hipError_t launch_predict(int n, int d, const uint16_t *h, const uint16_t *w1, const float *b1, const float *w2,
                          const float *b2, const float *w3, const float *b3, float *work, float *logit,
                          uint8_t *pred, hipStream_t s)
{
    const int row_tiles = (n + L1_TILE - 1) / L1_TILE;
    const int groups = (row_tiles + 7) / 8;  // rounds of 8 row tiles, one per XCD
    const int per_tile = KSPLIT * (SAE_PRED_H1 / L1_TILE);
    hipLaunchKernelGGL(k_pred_l1, dim3(groups * 8 * per_tile), dim3(L1_THREADS), 0, s, n, d, h, w1, work, row_tiles);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(k_pred_l23, dim3((n + L23_ROWS - 1) / L23_ROWS), dim3(L23_THREADS), 0, s, n, work, b1, w2, b2,
                       w3, b3, logit, pred);
    return hipGetLastError();
}
