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

    // Four register sets: the operands of a wave's step are loaded four of
    // its steps ahead.  Loads past the range re-read its last step (never a
    // load behind a branch, which would be waited for on the spot).
    constexpr int PD = 4;
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

// ---------------------------------------------------------------- fwd / dgrad
// Forward (and input gradient) of 1x1x1, stride-1 convolutions with at most
// 64 source and 64 target channels, as a streaming GEMM: a workgroup owns
// 256 voxels of one sample, loads all their source channels (16-byte loads of
// 8 voxels of one channel), transposes 8 x 8 blocks in registers into
// voxel-major rows of LDS (16-byte slot of channel group cg in voxel v at
// cg ^ (v & 7)), and each wave multiplies 64-voxel blocks by every target channel:
// A = the voxel rows (K = source channels), B = weight fragments from the
// prepared [K / 32][target][32] layout, which serves the forward (K = C_in)
// and the input gradient (K = C_out) alike.  An accumulator row block is four
// consecutive voxels of one target channel: stored as 8 bytes (old value
// added first when accumulating, one rounding).  HBM-bound: each source and
// target element moves once.
namespace {
struct PfArgs {
    const bf16* src;   // [N][Cs][V]
    const bf16* wt;    // [Cs / 32][Ct][32]
    const float* bias; // [Ct] or null
    bf16* dst;         // [N][Ct][V]
    int Cs, Ct;
    int64_t V;
    int64_t cpv;       // 256-voxel chunks per sample
    int accumulate;
};
constexpr int kPfVox = 256;
constexpr int kPfOutPitch = kPfVox * 2 + 16;  // bytes per target channel of a staged output tile
__device__ __forceinline__ uint32_t pf_lo(uint32_t lo, uint32_t hi) {
    return __builtin_amdgcn_perm(hi, lo, 0x05040100u);  // lo16(lo) | lo16(hi) << 16
}
__device__ __forceinline__ uint32_t pf_hi(uint32_t lo, uint32_t hi) {
    return __builtin_amdgcn_perm(hi, lo, 0x07060302u);  // hi16(lo) | hi16(hi) << 16
}
}  // namespace

__global__ __launch_bounds__(256) void conv_pw_fd(PfArgs a) {
    // one 256-voxel round: the staged output tile reuses the input rows
    static_assert(kPfVox == 256, "outputs are staged over the input tile");
    constexpr int kLds = kPfVox * 128 > 64 * kPfOutPitch ? kPfVox * 128 : 64 * kPfOutPitch;
    __shared__ __align__(16) unsigned char xs[kLds];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int64_t n = blockIdx.x / a.cpv;
    const int64_t v0 = (blockIdx.x - n * a.cpv) * kPfVox;
    const int ncg = a.Cs >> 3;  // source channel groups of 8
    // staging: thread (cg = tid % 8, voxel group g = tid / 8 + 32 r)
    const int cg = tid & 7;
    const bf16* sp = a.src + (n * a.Cs + (int64_t)cg * 8) * a.V;
#pragma unroll
    for (int r = 0; r < kPfVox / 8 / 32; ++r) {
        const int g = (tid >> 3) + 32 * r;
        const int64_t v = v0 + 8 * g;
        const bool live = cg < ncg && v < a.V;
        // idle or past-the-end items re-read the first group (never stored)
        const int64_t off = live ? v : 0;
        const int cgc = live ? 0 : -cg;  // keep the channel inside the tensor
        uint4 u[8];
#pragma unroll
        for (int j = 0; j < 8; ++j)
            u[j] = *reinterpret_cast<const uint4*>(sp + ((int64_t)cgc * 8 + j) * a.V + off);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int wd = e >> 1;
            uint32_t o[4];
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                const uint32_t wl = wd == 0 ? u[2 * c].x : wd == 1 ? u[2 * c].y
                                  : wd == 2 ? u[2 * c].z : u[2 * c].w;
                const uint32_t wh = wd == 0 ? u[2 * c + 1].x : wd == 1 ? u[2 * c + 1].y
                                  : wd == 2 ? u[2 * c + 1].z : u[2 * c + 1].w;
                o[c] = (e & 1) ? pf_hi(wl, wh) : pf_lo(wl, wh);
            }
            const int vl = 8 * g + e;
            *reinterpret_cast<uint4*>(xs + vl * 128 + ((cg ^ (vl & 7)) << 4)) =
                make_uint4(o[0], o[1], o[2], o[3]);
        }
    }
    __syncthreads();

    const int li = lane & 15, kg = lane >> 4;
    const int nks = a.Cs >> 5, nnt = a.Ct >> 4;
    bf16x8 B[2][4];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            // tiles past Cs / Ct re-read tile 0 (their sums are never used)
            const int kc = ks < nks ? ks : 0, nt = t < nnt ? t : 0;
            B[ks][t] = __builtin_bit_cast(
                bf16x8, *reinterpret_cast<const uint4*>(
                            a.wt + ((int64_t)(kc * a.Ct + nt * 16 + li) * 32 + kg * 8)));
        }
    // wave w multiplies voxels 256 rr + 64 w .. + 63 of the chunk
#pragma unroll 1
    for (int rr = 0; rr < kPfVox / 256; ++rr) {
        const int vb = rr * 256 + wave * 64;
        f32x4 acc[4][4];
#pragma unroll
        for (int m = 0; m < 4; ++m)
#pragma unroll
            for (int t = 0; t < 4; ++t) acc[m][t] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
            if (ks >= nks) break;
            bf16x8 A[4];
#pragma unroll
            for (int m = 0; m < 4; ++m) {
                const int vl = vb + m * 16 + li;
                const int c8 = ks * 4 + kg;
                A[m] = __builtin_bit_cast(
                    bf16x8,
                    *reinterpret_cast<const uint4*>(xs + vl * 128 + ((c8 ^ (vl & 7)) << 4)));
            }
#pragma unroll
            for (int m = 0; m < 4; ++m)
#pragma unroll
                for (int t = 0; t < 4; ++t)
                    acc[m][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(A[m], B[ks][t], acc[m][t],
                                                                       0, 0, 0);
        }
        // acc[m][t][j]: voxel v0 + vb + 16 m + 4 kg + j, target channel 16 t + li
        if (a.accumulate) {
            // old value added before the one rounding: stored from the lanes
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                if (t >= nnt) break;
                const int co = t * 16 + li;
                bf16* dp = a.dst + (n * a.Ct + co) * a.V;
#pragma unroll
                for (int m = 0; m < 4; ++m) {
                    const int64_t v = v0 + vb + m * 16 + kg * 4;
                    if (v >= a.V) continue;
                    uint2* q = reinterpret_cast<uint2*>(dp + v);
                    const uint2 o = *q;
                    const float r0 = acc[m][t][0] + __uint_as_float(o.x << 16);
                    const float r1 = acc[m][t][1] + __uint_as_float(o.x & 0xffff0000u);
                    const float r2 = acc[m][t][2] + __uint_as_float(o.y << 16);
                    const float r3 = acc[m][t][3] + __uint_as_float(o.y & 0xffff0000u);
                    *q = make_uint2(pack_bf16x2(r0, r1), pack_bf16x2(r2, r3));
                }
            }
            continue;
        }
        // staged through LDS as [target channel][voxel] rows, then stored as
        // 16-byte pieces of whole rows
        __syncthreads();  // every wave has read its operands of this round
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            if (t >= nnt) break;
            const int co = t * 16 + li;
            const float bv = a.bias ? a.bias[co] : 0.f;
#pragma unroll
            for (int m = 0; m < 4; ++m)
                *reinterpret_cast<uint2*>(xs + co * kPfOutPitch + (wave * 64 + m * 16 + kg * 4) * 2) =
                    make_uint2(pack_bf16x2(acc[m][t][0] + bv, acc[m][t][1] + bv),
                               pack_bf16x2(acc[m][t][2] + bv, acc[m][t][3] + bv));
        }
        __syncthreads();
        for (int it = tid; it < a.Ct * (256 / 8); it += 256) {
            const int co = it >> 5, pc = it & 31;
            const int64_t v = v0 + rr * 256 + pc * 8;
            if (v < a.V)
                *reinterpret_cast<uint4*>(a.dst + (n * a.Ct + co) * a.V + v) =
                    *reinterpret_cast<const uint4*>(xs + co * kPfOutPitch + pc * 16);
        }
    }
}

bool pw_fd_ok(const ConvGeom& g, rat3d_dtype dt, bool dgrad) {
    const int cs = dgrad ? g.Co : g.Ci, ct = dgrad ? g.Ci : g.Co;
    const int64_t V = (int64_t)g.D * g.H * g.W;
    return dt == RAT3D_BF16 && g.k == 1 && g.s == 1 && g.p == 0 && (cs == 32 || cs == 64) &&
           ct % 16 == 0 && ct <= 64 && V % 8 == 0;
}

rat3d_status conv_fd_pw(const ConvGeom& g, bool dgrad, const void* src, const void* wt,
                        const float* bias, void* dst, int accumulate, hipStream_t st) {
    PfArgs a;
    a.src = (const bf16*)src;
    a.wt = (const bf16*)wt;
    a.bias = dgrad ? nullptr : bias;
    a.dst = (bf16*)dst;
    a.Cs = dgrad ? g.Co : g.Ci;
    a.Ct = dgrad ? g.Ci : g.Co;
    a.V = (int64_t)g.D * g.H * g.W;
    a.cpv = ceil_div(a.V, kPfVox);
    a.accumulate = accumulate;
    const char* tag = dgrad ? (accumulate ? "conv_pw_dgrad_acc" : "conv_pw_dgrad") : "conv_pw_fwd";
    ProfScope ps(tag, st, conv_flops(g), conv_bytes(g, 2));
    conv_pw_fd<<<(unsigned)(g.N * a.cpv), 256, 0, st>>>(a);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
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
