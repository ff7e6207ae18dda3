// Weight gradient of 1x1x1, stride-1 convolutions as a plain GEMM:
// dw[co][ci] = sum over (n, v) of dy[n][co][v] * x[n][ci][v].  In NCDHW both
// operands are rows that are contiguous in the reduction index v, so every
// MFMA operand (8 consecutive voxels of one channel) is one 16-byte global
// load; no LDS staging is needed.  The voxel range is split over workgroups;
// inside a workgroup the four waves take interleaved 32-voxel steps, their
// 64 x 64 partial tiles are summed through LDS in wave order, and the
// workgroup's tile goes to the workspace for the fixed-order reduction.
#include "common.hpp"
#include "kernels.hpp"
#include "prof.hpp"

namespace rat3d {

namespace {
union F16B {
    uint4 u;
    bf16x8 b;
};

struct PwArgs {
    const bf16* x;   // [N][Ci][V]
    const bf16* dy;  // [N][Co][V]
    float* part;     // [splits][Co][Ci]
    int N, Ci, Co;
    int64_t V;
    int64_t steps;       // 32-voxel steps in total (N * V / 32)
    int64_t per_split;   // steps per workgroup
};
}  // namespace

__global__ __launch_bounds__(256) void conv_pw_wgrad(PwArgs a) {
    __shared__ float red[4][64 * 64];  // each wave's 64 x 64 partial tile
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int li = lane & 15, kg = lane >> 4;
    const int co0 = blockIdx.y * 64, ci0 = blockIdx.z * 64;
    const int nco = min(64, a.Co - co0) / 16, nci = min(64, a.Ci - ci0) / 16;
    const int64_t s_beg = (int64_t)blockIdx.x * a.per_split;
    const int64_t s_end = s_beg + a.per_split < a.steps ? s_beg + a.per_split : a.steps;
    const int64_t spp = a.V / 32;  // steps per (n) plane

    f32x4 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    // Channel tiles past the tensor re-read its last channel: their sums are
    // never stored, and no load sits behind a branch.
    auto load = [&](int64_t st, F16B (&av)[4], F16B (&bv)[4]) {
        const int64_t n = st / spp;
        const int64_t v = (st - n * spp) * 32 + kg * 8;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int co = min(co0 + t * 16 + li, a.Co - 1), ci = min(ci0 + t * 16 + li, a.Ci - 1);
            av[t].u = *reinterpret_cast<const uint4*>(a.dy + ((int64_t)n * a.Co + co) * a.V + v);
            bv[t].u = *reinterpret_cast<const uint4*>(a.x + ((int64_t)n * a.Ci + ci) * a.V + v);
        }
    };

    // Three register sets: the operands of a wave's step are loaded three of
    // its steps ahead.  Loads past the range re-read its last step (never a
    // load behind a branch, which would be waited for on the spot).
    constexpr int PD = 3;
    F16B av[PD][4], bv[PD][4];
    const int64_t last = s_end - 1;
#pragma unroll
    for (int r = 0; r < PD; ++r) {
        const int64_t sr = s_beg + wave + 4 * r;
        load(sr < s_end ? sr : last, av[r], bv[r]);
    }
    for (int64_t st = s_beg + wave; st < s_end; st += 4 * PD) {
#pragma unroll
        for (int r = 0; r < PD; ++r) {
            const int64_t sc = st + 4 * r;
            if (sc < s_end) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av[r][i].b, bv[r][j].b,
                                                                           acc[i][j], 0, 0, 0);
            }
            const int64_t sn = sc + 4 * PD;
            load(sn < s_end ? sn : last, av[r], bv[r]);
        }
    }

    // acc[i][j][e]: co = co0 + 16i + 4kg + e, ci = ci0 + 16j + li
    float* mine = red[wave];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e) mine[(16 * i + 4 * kg + e) * 64 + 16 * j + li] = acc[i][j][e];
    __syncthreads();
    float* out = a.part + (int64_t)blockIdx.x * a.Co * a.Ci;
    for (int e = tid; e < 64 * 64; e += 256) {
        const int r = e >> 6, c = e & 63;
        if (r >= nco * 16 || c >= nci * 16) continue;
        const float s = ((red[0][e] + red[1][e]) + red[2][e]) + red[3][e];
        out[(int64_t)(co0 + r) * a.Ci + ci0 + c] = s;
    }
}

bool pw_wgrad_ok(const ConvGeom& g, rat3d_dtype dt) {
    const int64_t V = (int64_t)g.D * g.H * g.W;
    return dt == RAT3D_BF16 && g.k == 1 && g.s == 1 && g.p == 0 && g.Ci % 16 == 0 &&
           g.Co % 16 == 0 && V % 32 == 0;
}

static int pw_splits(const ConvGeom& g) {
    const int64_t steps = (int64_t)g.N * g.D * g.H * g.W / 32;
    const int64_t tiles = ceil_div(g.Co, 64) * ceil_div(g.Ci, 64);
    int64_t s = ceil_div(2 * device_cus(), tiles);  // two workgroups per CU (LDS)
    if (s > steps) s = steps;
    if (s < 1) s = 1;
    return (int)s;
}

size_t pw_wgrad_ws(const ConvGeom& g) {
    return (size_t)pw_splits(g) * g.Co * g.Ci * sizeof(float);
}

rat3d_status conv_wgrad_pw(const ConvGeom& g, const void* x, const void* dy, float* dw,
                           int accumulate, void* ws, hipStream_t st) {
    PwArgs a;
    a.x = (const bf16*)x;
    a.dy = (const bf16*)dy;
    a.part = (float*)ws;
    a.N = g.N;
    a.Ci = g.Ci;
    a.Co = g.Co;
    a.V = (int64_t)g.D * g.H * g.W;
    a.steps = (int64_t)g.N * a.V / 32;
    const int S = pw_splits(g);
    a.per_split = ceil_div(a.steps, S);
    const int Sreal = (int)ceil_div(a.steps, a.per_split);
    {
        ProfScope ps("conv_pw_wgrad", st, conv_flops(g), conv_bytes(g, 2));
        conv_pw_wgrad<<<dim3(Sreal, (unsigned)ceil_div(g.Co, 64), (unsigned)ceil_div(g.Ci, 64)),
                        256, 0, st>>>(a);
        RAT3D_LAUNCH_CHECK();
    }
    const int64_t count = (int64_t)g.Co * g.Ci;
    ProfScope ps("wgrad_reduce", st, 0.0, 4.0 * count * (Sreal + 1 + accumulate));
    return wgrad_reduce_launch(a.part, Sreal, count, dw, accumulate, st);
}

}  // namespace rat3d
