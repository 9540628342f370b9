// Multi-turn session predictor (Sec. 3.3): y = W3 relu(W2 relu(W1 h + b1) + b2) + b3
// over a batch of last-token hidden states, on the matrix cores.
//
// Layer 1 (n x d) . (d x 256) is the one dense contraction of the method:
// bf16 products (exact) summed in fp32 by v_mfma_f32_32x32x16_bf16.  A
// workgroup of 8 waves (two per SIMD, so that one issues MFMAs while the other
// waits on LDS or the barrier) computes a 128 x 128 tile, each wave 64 rows x
// 32 columns (two 32 x 32 blocks).
// The sum over k is order-free, so A and B may share any permutation of k:
// lane l (row / column l mod 32, half l / 32) supplies, in a 64-wide k step,
// the 32 contiguous values of its half (64 bytes, four 16-byte loads), and
// MFMA m of the step takes values 8m .. 8m + 7 of both operands.  The next
// step's loads are issued before this step's four MFMAs.  Tiles are ordered
// so that the four column tiles of a row tile land on the same XCD (block
// ids go round-robin over the 8 XCDs) and read the same hidden-state rows
// through one L2.
//
// Layers 2 and 3 are fp32: v_mfma_f32_16x16x4f32 for (16 rows x 256) . (256 x
// 64) in a workgroup of 8 waves (each a k eighth of all 16 rows, loaded once
// and fed to the four 16-column blocks, every load of a wave issued at once,
// the eighths summed in a fixed order), then the 64-term layer 3 by shuffles.  Layer 1's four k
// slices are added here, in slice order, before b1 and the ReLU.
#include <mutex>

#include "sae_internal.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int L1_TILE = 128;       // rows and columns of a workgroup's tile

constexpr int L1_THREADS = 512;  // 8 waves, each 64 x 32 (2 x 1 MFMA blocks of 32 x 32)
constexpr int L1_RPT = L1_TILE / (L1_THREADS / 8);  // tile rows a thread moves per step (2)

constexpr int KSTEP = 64;          // k per step
constexpr int KSPLIT = 4;          // k slices (workgroups per tile); their sums meet in layer 2
constexpr int L1_NS = 2;           // steps in flight in registers (even; 4 measured slower)
constexpr int LDS_ROW16 = 9;       // LDS row of a tile: 128 bytes of k + 16 bytes of padding
constexpr int L23_THREADS = 512;   // 8 waves: one k eighth each, both layer-2 column halves
constexpr int L23_ROWS = 16;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v)
{
    bf16x8 r;
    __builtin_memcpy(&r, &v, sizeof(r));
    return r;
}

// One step (64 k) of a thread's share of the A and B tiles: rows j = 0, 1.
struct Stage {
    uint4 a0, a1, b0, b1;
};

__device__ __forceinline__ void load_stage(Stage &x, const uint4 *ga0, const uint4 *ga1, const uint4 *gb0,
                                           long long bstride, int step, int nsteps)
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
    x.b0 = m(gb0[o]);
    x.b1 = m(gb0[bstride + o]);
}

__device__ __forceinline__ void put_stage(const Stage &x, uint4 *la, uint4 *lb, int ls, int lstride)
{
    la[ls] = x.a0;
    la[ls + lstride] = x.a1;
    lb[ls] = x.b0;
    lb[ls + lstride] = x.b1;
}

// The 8 MFMAs of one step for a wave's 64 x 32 block (2 x 1 blocks).
__device__ __forceinline__ void mfma_step(floatx16 (&acc)[2], const uint4 *tla, const uint4 *tlb, int wr, int wc,
                                          int orow, int och)
{
    const uint4 *la = tla + (wr * 64 + orow) * LDS_ROW16 + och;
    const uint4 *lb = tlb + (wc * 32 + orow) * LDS_ROW16 + och;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        const bf16x8 a0 = as_bf16x8(la[m]), a1 = as_bf16x8(la[32 * LDS_ROW16 + m]);
        const bf16x8 b0 = as_bf16x8(lb[m]);
        acc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a0, b0, acc[0], 0, 0, 0);
        acc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a1, b0, acc[1], 0, 0, 0);
    }
}

// One workgroup per compute unit (its LDS alone rules out three), two waves
// per SIMD.
__global__ void __launch_bounds__(L1_THREADS) __attribute__((amdgpu_waves_per_eu(2, 2)))
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
    const int wr = wave >> 2, wc = wave & 3;           // this wave's 64 rows x 32 columns
    const int kper = d / KSPLIT;                       // a multiple of 64
    const int kbeg = ks * kper, nsteps = kper / KSTEP;
    // global -> LDS: thread t moves 16-byte chunks of rows t / 8 + 64 j (j < 2),
    // chunk t mod 8 of each row's 128 bytes, of both tiles
    static_assert(L1_RPT == 2, "two tile rows per thread and step");
    const int lr = tid >> 3, lc = tid & 7;
    const uint4 *ga0, *ga1;
    {
        auto arow = [&](int j) {
            int r = rt * L1_TILE + lr + 64 * j;
            r = r < n ? r : n - 1;  // rows past n repeat row n - 1 (results dropped)
            return reinterpret_cast<const uint4 *>(h + (long long)r * d + kbeg) + lc;
        };
        ga0 = arow(0);
        ga1 = arow(1);
    }
    const uint4 *gb0 = reinterpret_cast<const uint4 *>(w1 + (long long)(ct * L1_TILE + lr) * d + kbeg) + lc;
    const long long bstride = 64ll * d / 8;  // 64 rows of W1, in uint4
    const int ls = lr * LDS_ROW16 + lc, lstride = 64 * LDS_ROW16;
    floatx16 acc[2];
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int i = 0; i < 16; ++i) acc[bi][i] = 0.0f;
    // operand reads: lane (row / column l mod 32, half l / 32) takes, in MFMA
    // m of a step, the 16 bytes at k = 32 half + 8 m of its row
    const int orow = lane & 31, och = (lane >> 5) * 4;
    // pipeline: step s is in LDS buffer s mod 2 while steps s + 1 .. s + L1_NS
    // are in flight in L1_NS register stages (the loop is unrolled by L1_NS so
    // that each stage is a fixed set of registers; a step past the end is all
    // zeros).  Step t >= 1 travels in stage (t - 1) mod L1_NS.
    Stage sg[L1_NS];
    load_stage(sg[0], ga0, ga1, gb0, bstride, 0, nsteps);
    put_stage(sg[0], lds[0][0], lds[0][1], ls, lstride);
#pragma unroll
    for (int j = 0; j < L1_NS; ++j) load_stage(sg[j], ga0, ga1, gb0, bstride, 1 + j, nsteps);
    __syncthreads();
    for (int st = 0; st < nsteps; st += L1_NS) {
#pragma unroll
        for (int j = 0; j < L1_NS; ++j) {
            const int b = j & 1;  // st is a multiple of L1_NS (even)
            mfma_step(acc, lds[b][0], lds[b][1], wr, wc, orow, och);                  // step st + j
            put_stage(sg[j], lds[b ^ 1][0], lds[b ^ 1][1], ls, lstride);              // step st + j + 1
            load_stage(sg[j], ga0, ga1, gb0, bstride, st + j + 1 + L1_NS, nsteps);
            __syncthreads();
        }
    }
    // partial sums of this k slice; C layout: lane l holds column l mod 32,
    // rows 8 (i / 4) + 4 (l / 32) + i mod 4 of each 32 x 32 block
    float *out = part + (long long)ks * n * SAE_PRED_H1;
    const int col = ct * L1_TILE + wc * 32 + (lane & 31);
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int i = 0; i < 16; ++i) {
            const int r = rt * L1_TILE + wr * 64 + bi * 32 + (i >> 2) * 8 + (lane >> 5) * 4 + (i & 3);
            if (r < n) out[(long long)r * SAE_PRED_H1 + col] = acc[bi][i];
        }
}

__global__ void __launch_bounds__(L23_THREADS) __attribute__((amdgpu_waves_per_eu(1, 2)))
k_pred_l23(int n, const float *part, const float *b1, const float *w2, const float *b2, const float *w3,
           const float *b3, float *logit, uint8_t *pred)
{
    // 16 rows per workgroup (every compute unit busy); wave w owns k eighth w
    // (32 of the 256 layer-1 units) of all 16 rows: it loads those units once
    // (four slices) and feeds them to the MFMAs of the four 16-column blocks
    // of layer 2; the eighths meet in LDS and are added in eighth order
    constexpr int NW = L23_THREADS / SAE_WAVE;  // 8
    constexpr int KW = SAE_PRED_H1 / NW;         // 32
    constexpr int NCB = SAE_PRED_H2 / 16;        // 4 column blocks
    __shared__ float hsum[NW - 1][NCB * 4][SAE_WAVE];
    __shared__ float ysum[L23_ROWS];
    const int lane = (int)__lane_id(), wave = threadIdx.x / SAE_WAVE;
    const int r0 = blockIdx.x * L23_ROWS;
    const int row = r0 + (lane & 15);
    const int rowc = row < n ? row : n - 1;
    const int grp = lane >> 4;
    // lane group g supplies k = 32 w + 8 g + s in MFMA s, for both operands
    // (v_mfma_f32_16x16x4f32: lane l gives A[l mod 16][l / 16] and
    // B[l / 16][l mod 16]); the layer-1 value is the sum of its k slices in
    // slice order, plus b1, ReLU
    const int kb = wave * KW + grp * 8;
    const long long slice = (long long)n * SAE_PRED_H1 / 4;  // in float4
    const float4 *pa = reinterpret_cast<const float4 *>(part + (long long)rowc * SAE_PRED_H1 + kb);
    const float4 *pc = reinterpret_cast<const float4 *>(b1 + kb);
    float4 v[KSPLIT][2], bw[NCB][2], c[2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {  // every load of the wave in flight together
#pragma unroll
        for (int q = 0; q < KSPLIT; ++q) v[q][u] = pa[q * slice + u];
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
            bw[cb][u] = reinterpret_cast<const float4 *>(w2 + (long long)(cb * 16 + (lane & 15)) * SAE_PRED_H1 + kb)[u];
        c[u] = pc[u];
    }
    __builtin_amdgcn_sched_barrier(0);
    floatx4 acc[NCB];
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
        for (int i = 0; i < 4; ++i) acc[cb][i] = 0.0f;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
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
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, bw[cb][u].x, acc[cb], 0, 0, 0);
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, bw[cb][u].y, acc[cb], 0, 0, 0);
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, bw[cb][u].z, acc[cb], 0, 0, 0);
            acc[cb] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, bw[cb][u].w, acc[cb], 0, 0, 0);
        }
    }
    // C layout: lane l holds column 16 cb + l mod 16, rows 4 (l / 16) + i
    if (wave > 0) {
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
            for (int i = 0; i < 4; ++i) hsum[wave - 1][cb * 4 + i][lane] = acc[cb][i];
    }
    __syncthreads();
    if (wave == 0) {
        // layer 2 complete (eighths in order); layer 3: each lane's four
        // columns' weights times relu(h2) for its 4 rows, then the sum over
        // the 16 lanes that share those rows
        float t[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) t[i] = 0.0f;
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb) {
            const int col = cb * 16 + (lane & 15);
            const float bias = b2[col], wt = w3[col];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                float h2 = acc[cb][i];
#pragma unroll
                for (int q = 0; q < NW - 1; ++q) h2 = h2 + hsum[q][cb * 4 + i][lane];
                h2 = h2 + bias;
                t[i] = t[i] + wt * (h2 > 0.0f ? h2 : 0.0f);
            }
        }
#pragma unroll
        for (int o = 1; o < 16; o <<= 1)
#pragma unroll
            for (int i = 0; i < 4; ++i) t[i] = t[i] + __shfl_xor(t[i], o);
        if ((lane & 15) == 0) {
#pragma unroll
            for (int i = 0; i < 4; ++i) ysum[grp * 4 + i] = t[i];
        }
    }
    __syncthreads();
    if (threadIdx.x < L23_ROWS) {
        const int r = r0 + threadIdx.x;
        const float y = ysum[threadIdx.x] + b3[0];
        if (r < n) {
            logit[r] = y;
            if (pred) pred[r] = y > 0.0f ? 1 : 0;
        }
    }
}

}  // namespace

// Layer 1's partial sums for sae_predict_sessions_noalloc: device memory of the
// library's own (each GPU holds its own copy of the array until the process
// ends).  Host code never passes `scratch` itself to a kernel (on the host it
// is only a stand-in for the symbol); it passes the device address that
// hipGetSymbolAddress returned for the current device.
static __device__ __align__(256) float scratch[(size_t)KSPLIT * SAE_PRED_NOALLOC_MAX_N * SAE_PRED_H1];

// The device address of `scratch` on the current device, looked up with that
// device current on its first use and kept per device.
hipError_t predict_scratch(float **out)
{
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void *addr[kMaxDevices] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *out = static_cast<float *>(addr[dev]);
    return hipSuccess;
}

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
