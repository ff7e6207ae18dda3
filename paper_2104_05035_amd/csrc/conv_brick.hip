// LDS-brick implicit-GEMM convolution for the dominant shapes: bfloat16,
// stride 1, cubic kernel 3 (pad 1) or 1 (pad 0), channel counts multiple of
// 32 (forward / input gradient) or 16/64 (weight gradient).
//
// Forward (and the stride-1 input gradient, which is the forward convolution
// of dy with the flipped, transposed weights): a workgroup computes an output
// tile of 4 x 8 x 16 voxels for 32 or 64 output channels.  For each chunk of
// 32 input channels it stages the halo'd input brick into LDS with the
// channel index innermost (64 bytes per voxel, four 16-byte groups of eight
// channels, XOR-swizzled by voxel so that the sixteen lanes of an MFMA row
// group hit distinct banks).  The GEMM K index is (tap, channel): for a tap,
// an MFMA A-operand row is one output voxel and its eight K values are eight
// consecutive channels of the shifted input voxel -- one 16-byte LDS read.
// B operands come from a weight copy pre-arranged as
// [chunk][tap][C_out][32 channels], so a lane's operand is one coalesced
// 16-byte global load (L1/L2 resident: every workgroup reads the same
// weights).  Each wave owns one output depth slice: 8 rows of 16 voxels by
// all output channels of the workgroup, i.e. 8 x (2 or 4) MFMA 16x16 tiles,
// and reuses each weight fragment across its 8 rows.
//
// Weight gradient: a workgroup owns dw for 64 output channels x 16 input
// channels x 27 taps (the four waves split the taps) and sums over a range
// of 2 x 8 x 16 output-voxel bricks.  GEMM K = voxels: the A operand (dy,
// 16 output channels x 32 voxels) is read straight from global memory as
// 16-byte rows of the NCDHW tensor; the B operand (x shifted by the tap) is
// read from LDS, where the input brick is kept as three copies pre-shifted
// by kw = 0, 1, 2 so that every 8-voxel operand row is 16-byte aligned.
// Partial tiles go to the workspace and are reduced in a fixed order.
//
// Grid mapping is XCD-aware: consecutive workgroup ids are dealt round-robin
// to the 8 XCDs, so ids are remapped to give each XCD a contiguous range of
// tiles (neighbouring bricks share halo lines in that XCD's L2).
#include "common.hpp"
#include "kernels.hpp"
#include "prof.hpp"

namespace rat3d {

namespace {

union F16B {
    uint4 u;
    bf16x8 b;
};

constexpr int kBD = 4, kBH = 8, kBW = 16;     // forward output tile
constexpr int kWD = 2, kWH = 8, kWW = 16;     // weight-gradient voxel brick

__device__ __forceinline__ f32x4 mfma(const F16B& a, const F16B& b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.b, b.b, c, 0, 0, 0);
}

struct FdArgs {
    const bf16* src;   // [N][Cs][D][H][W]
    const bf16* wt;    // [Cs/32][KT][Ct][32]
    const float* bias; // [Ct] or null
    bf16* dst;         // [N][Ct][D][H][W]
    int N, Cs, Ct, D, H, W;
    int td, th, tw;    // tiles per axis
    int accumulate;
};

}  // namespace

// ---------------------------------------------------------------- weight prep
// fwd:   wt[((c/32)*KT + t)*Co + co]*32 + c%32] = w[co][c][t]
__global__ void prep_fwd_weights(const bf16* __restrict__ w, int Co, int Ci, int KT,
                                 bf16* __restrict__ wt) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t total = (int64_t)Co * Ci * KT;
    if (i >= total) return;
    const int t = (int)(i % KT);
    const int c = (int)((i / KT) % Ci);
    const int co = (int)(i / ((int64_t)KT * Ci));
    wt[(((int64_t)(c >> 5) * KT + t) * Co + co) * 32 + (c & 31)] = w[i];
}

// dgrad: wt[((co/32)*KT + t)*Ci + ci]*32 + co%32] = w[co][ci][KT - 1 - t]
__global__ void prep_dgrad_weights(const bf16* __restrict__ w, int Co, int Ci, int KT,
                                   bf16* __restrict__ wt) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t total = (int64_t)Co * Ci * KT;
    if (i >= total) return;
    const int t = (int)(i % KT);
    const int ci = (int)((i / KT) % Ci);
    const int co = (int)(i / ((int64_t)KT * Ci));
    wt[(((int64_t)(co >> 5) * KT + (KT - 1 - t)) * Ci + ci) * 32 + (co & 31)] = w[i];
}

// ---------------------------------------------------------------- fwd / dgrad
template <int KS, int NT>
__global__ __launch_bounds__(256, 2) void conv_brick_fd(FdArgs a) {
    constexpr int P = (KS - 1) / 2;
    constexpr int PD = kBD + KS - 1, PH = kBH + KS - 1, PW = kBW + KS - 1;
    constexpr int NV = PD * PH * PW;
    constexpr int KT = KS * KS * KS;
    __shared__ uint4 brick[NV * 4];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int L = xcd_remap(blockIdx.x, gridDim.x);
    const int tw = L % a.tw;
    int r = L / a.tw;
    const int th = r % a.th;
    r /= a.th;
    const int td = r % a.td;
    const int n = r / a.td;
    const int d0 = td * kBD, h0 = th * kBH, w0 = tw * kBW;
    const int co0 = blockIdx.y * NT * 16;
    const int64_t HW = (int64_t)a.H * a.W, V = HW * a.D;

    f32x4 acc[8][NT];
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

    const int li = lane & 15, kg = lane >> 4;
    for (int c0 = 0; c0 < a.Cs; c0 += 32) {
        __syncthreads();
        if (a.W % 4 == 0) {
            // item = (channel group, brick row, aligned 4-wide column group):
            // eight 8-byte loads (one per channel) give 4 voxels x 8 channels
            constexpr int GS0 = -4 * ((P + 3) / 4);          // first group, relative to w0
            constexpr int NG = (PW - P - GS0 + 3) / 4;       // groups covering the brick row
            for (int it = tid; it < 4 * PD * PH * NG; it += 256) {
                const int q = it % NG;
                const int rr = it / NG;
                const int row = rr % (PD * PH), cg = rr / (PD * PH);
                const int hh = row % PH, dd = row / PH;
                const int d = d0 - P + dd, h = h0 - P + hh, wg = w0 + GS0 + 4 * q;
                uint2 v[8];
                if ((unsigned)d < (unsigned)a.D && (unsigned)h < (unsigned)a.H &&
                    (unsigned)wg < (unsigned)a.W) {
                    const bf16* p = a.src + ((int64_t)n * a.Cs + c0 + cg * 8) * V + d * HW +
                                    (int64_t)h * a.W + wg;
#pragma unroll
                    for (int j = 0; j < 8; ++j) v[j] = *reinterpret_cast<const uint2*>(p + j * V);
                } else {
#pragma unroll
                    for (int j = 0; j < 8; ++j) v[j] = make_uint2(0u, 0u);
                }
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int ww = wg + e - (w0 - P);
                    if (ww < 0 || ww >= PW) continue;
                    const int vox = (dd * PH + hh) * PW + ww;
                    uint32_t c[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const uint32_t word = (e < 2) ? v[j].x : v[j].y;
                        c[j] = (e & 1) ? (word >> 16) : (word & 0xffffu);
                    }
                    brick[vox * 4 + (cg ^ ((vox >> 1) & 3))] =
                        make_uint4(c[0] | (c[1] << 16), c[2] | (c[3] << 16), c[4] | (c[5] << 16),
                                   c[6] | (c[7] << 16));
                }
            }
        } else {
            // item = (channel group, brick voxel), voxel fastest
            for (int it = tid; it < NV * 4; it += 256) {
                const int vox = it % NV, cg = it / NV;
                const int ww = vox % PW, rr = vox / PW;
                const int hh = rr % PH, dd = rr / PH;
                const int d = d0 - P + dd, h = h0 - P + hh, w = w0 - P + ww;
                uint4 pk = make_uint4(0u, 0u, 0u, 0u);
                if ((unsigned)d < (unsigned)a.D && (unsigned)h < (unsigned)a.H &&
                    (unsigned)w < (unsigned)a.W) {
                    const bf16* p = a.src + ((int64_t)n * a.Cs + c0 + cg * 8) * V + d * HW +
                                    (int64_t)h * a.W + w;
                    uint32_t v[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) v[j] = p[j * V];
                    pk.x = v[0] | (v[1] << 16);
                    pk.y = v[2] | (v[3] << 16);
                    pk.z = v[4] | (v[5] << 16);
                    pk.w = v[6] | (v[7] << 16);
                }
                brick[vox * 4 + (cg ^ ((vox >> 1) & 3))] = pk;
            }
        }
        __syncthreads();
        const bf16* wc = a.wt + (int64_t)(c0 >> 5) * KT * a.Ct * 32;
        // weight fragments are double-buffered: tap t+1 loads while tap t multiplies
        F16B bc[NT];
#pragma unroll
        for (int ct = 0; ct < NT; ++ct)
            bc[ct].u = *reinterpret_cast<const uint4*>(wc + ((int64_t)(co0 + ct * 16 + li)) * 32 +
                                                        kg * 8);
#pragma unroll 1
        for (int tap = 0; tap < KT; ++tap) {
            const int kd = tap / (KS * KS), kh = (tap / KS) % KS, kw = tap % KS;
            F16B bn[NT];
            const int tn = tap + 1 < KT ? tap + 1 : tap;
#pragma unroll
            for (int ct = 0; ct < NT; ++ct)
                bn[ct].u = *reinterpret_cast<const uint4*>(
                    wc + ((int64_t)tn * a.Ct + co0 + ct * 16 + li) * 32 + kg * 8);
#pragma unroll
            for (int rw = 0; rw < 8; ++rw) {
                const int vox = ((wave + kd) * PH + (rw + kh)) * PW + li + kw;
                F16B av;
                av.u = brick[vox * 4 + (kg ^ ((vox >> 1) & 3))];
#pragma unroll
                for (int ct = 0; ct < NT; ++ct) acc[rw][ct] = mfma(av, bc[ct], acc[rw][ct]);
            }
#pragma unroll
            for (int ct = 0; ct < NT; ++ct) bc[ct] = bn[ct];
        }
    }

    // epilogue: lane holds 4 consecutive w of one output channel per tile
    const int d = d0 + wave;
    if (d >= a.D) return;
    const bool full_w = (w0 + kBW <= a.W) && ((a.W & 3) == 0);
#pragma unroll
    for (int rw = 0; rw < 8; ++rw) {
        const int h = h0 + rw;
        if (h >= a.H) continue;
#pragma unroll
        for (int ct = 0; ct < NT; ++ct) {
            const int co = co0 + ct * 16 + li;
            const float bv = a.bias ? a.bias[co] : 0.f;
            const int w = w0 + 4 * kg;
            bf16* q = a.dst + ((int64_t)n * a.Ct + co) * V + d * HW + (int64_t)h * a.W + w;
            float v[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = acc[rw][ct][e] + bv;
            if (full_w) {
                uint2* q2 = reinterpret_cast<uint2*>(q);
                if (a.accumulate) {
                    const uint2 o = *q2;
                    v[0] += __uint_as_float(o.x << 16);
                    v[1] += __uint_as_float(o.x & 0xffff0000u);
                    v[2] += __uint_as_float(o.y << 16);
                    v[3] += __uint_as_float(o.y & 0xffff0000u);
                }
                *q2 = make_uint2((uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16),
                                 (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16));
            } else {
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    if (w + e >= a.W) break;
                    float o = v[e];
                    if (a.accumulate) o += bf2f(q[e]);
                    q[e] = f2bf(o);
                }
            }
        }
    }
}

// ---------------------------------------------------------------- wgrad
namespace {
struct WgArgs {
    const bf16* x;   // [N][Ci][D][H][W]
    const bf16* dy;  // [N][Co][D][H][W]
    float* part;     // [ranges][Co][Ci][KT]
    int N, Ci, Co, D, H, W;
    int td, th, tw;  // bricks per axis
    int64_t nbricks;
    int bpr;         // bricks per range
    int cigs, cogs;  // input-channel groups of 16, output-channel groups of 64
};
}  // namespace

// Partials are stored in the accumulators' register order: per workgroup a
// block of kWgPart floats, element ((j * 4 + ct) * 4 + e) * 256 + tid, so every
// store instruction writes 256 contiguous bytes.  wgrad_brick_reduce sums the
// ranges in order and scatters each sum to its (co, ci, tap).
constexpr int kWgNtap = 7;                       // taps per wave: wave + 4 j < 27
constexpr int kWgPart = kWgNtap * 4 * 4 * 256;   // floats per workgroup partial

template <int KS>
__global__ __launch_bounds__(256, 2) void conv_brick_wgrad(WgArgs a) {
    constexpr int P = (KS - 1) / 2;
    constexpr int KT = KS * KS * KS;
    static_assert(KS == 3, "the weight-gradient brick assembles kw = 0, 1, 2 copies");
    constexpr int PD = kWD + KS - 1, PH = kWH + KS - 1;
    constexpr int ROWS = PD * PH;
    constexpr int CIS = ROWS * 32 + 16;  // bytes per input channel (rows of 16 bf16) + pad
    constexpr int KWS = 16 * CIS;        // bytes per kw-shifted copy
    constexpr int NTAP = (KT + 3) / 4;   // taps per wave
    static_assert(NTAP == kWgNtap, "partial layout");
    constexpr int NIT = (16 * ROWS + 255) / 256;  // staging items per thread
    __shared__ __align__(16) unsigned char xs[KS * KWS];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int L = xcd_remap(blockIdx.x, gridDim.x);
    const int cig = L % a.cigs;
    const int rest = L / a.cigs;
    const int cog = rest % a.cogs;
    const int range = rest / a.cogs;
    const int ci0 = cig * 16, co0 = cog * 64;
    const int64_t b_beg = (int64_t)range * a.bpr;
    const int64_t b_end = b_beg + a.bpr < a.nbricks ? b_beg + a.bpr : a.nbricks;
    const int64_t HW = (int64_t)a.H * a.W, V = HW * a.D;
    const int li = lane & 15, kg = lane >> 4;
    const int hl_l = kg >> 1, wl = (kg & 1) * 8;

    f32x4 acc[NTAP][4];
#pragma unroll
    for (int j = 0; j < NTAP; ++j)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[j][c] = f32x4{0.f, 0.f, 0.f, 0.f};

    struct Brick {
        int n, d0, h0, w0;
    };
    auto brick_at = [&](int64_t b) {
        Brick k;
        k.w0 = (int)(b % a.tw) * kWW;
        int64_t r = b / a.tw;
        k.h0 = (int)(r % a.th) * kWH;
        r /= a.th;
        k.d0 = (int)(r % a.td) * kWD;
        k.n = (int)(r / a.td);
        return k;
    };

    // Staging item = (input channel, brick row): the row's 16 aligned voxels
    // (two 16-byte loads) plus one halo voxel on each side, held in registers
    // m[0] = (?, x[w0-1]), m[1..8] = x[w0 .. w0+15], m[9] = (x[w0+16], ?).
    // The next brick's rows are fetched before the current brick's K loop so
    // that the loads are in flight while the MFMAs run.
    uint32_t m[NIT][10];
    auto fetch = [&](const Brick& k) {
#pragma unroll
        for (int q = 0; q < NIT; ++q) {
#pragma unroll
            for (int j = 0; j < 10; ++j) m[q][j] = 0u;
            const int it = tid + 256 * q;
            if (it >= 16 * ROWS) continue;
            const int row = it % ROWS, ci = it / ROWS;
            const int d = k.d0 - P + row / PH, h = k.h0 - P + row % PH;
            if ((unsigned)d >= (unsigned)a.D || (unsigned)h >= (unsigned)a.H) continue;
            const bf16* p = a.x + ((int64_t)k.n * a.Ci + ci0 + ci) * V + d * HW +
                            (int64_t)h * a.W + k.w0;
            if (k.w0 + 8 <= a.W) {
                const uint4 u = *reinterpret_cast<const uint4*>(p);
                m[q][1] = u.x; m[q][2] = u.y; m[q][3] = u.z; m[q][4] = u.w;
            }
            if (k.w0 + 16 <= a.W) {
                const uint4 u = *reinterpret_cast<const uint4*>(p + 8);
                m[q][5] = u.x; m[q][6] = u.y; m[q][7] = u.z; m[q][8] = u.w;
            }
            if (k.w0 >= 1) m[q][0] = (uint32_t)p[-1] << 16;
            if (k.w0 + 16 < a.W) m[q][9] = (uint32_t)p[16];
        }
    };
    // copy kw holds input columns w0 - 1 + kw ... as aligned 16-byte LDS rows
    auto commit = [&]() {
#pragma unroll
        for (int q = 0; q < NIT; ++q) {
            const int it = tid + 256 * q;
            if (it >= 16 * ROWS) continue;
            const int row = it % ROWS, ci = it / ROWS;
            unsigned char* base = xs + ci * CIS + row * 32;
            *reinterpret_cast<uint4*>(base + KWS) = make_uint4(m[q][1], m[q][2], m[q][3], m[q][4]);
            *reinterpret_cast<uint4*>(base + KWS + 16) =
                make_uint4(m[q][5], m[q][6], m[q][7], m[q][8]);
            uint32_t s0[8], s2[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                s0[i] = (m[q][i] >> 16) | (m[q][i + 1] << 16);
                s2[i] = (m[q][i + 1] >> 16) | (m[q][i + 2] << 16);
            }
            *reinterpret_cast<uint4*>(base) = make_uint4(s0[0], s0[1], s0[2], s0[3]);
            *reinterpret_cast<uint4*>(base + 16) = make_uint4(s0[4], s0[5], s0[6], s0[7]);
            *reinterpret_cast<uint4*>(base + 2 * KWS) = make_uint4(s2[0], s2[1], s2[2], s2[3]);
            *reinterpret_cast<uint4*>(base + 2 * KWS + 16) =
                make_uint4(s2[4], s2[5], s2[6], s2[7]);
        }
    };

    if (b_beg < b_end) fetch(brick_at(b_beg));
    for (int64_t b = b_beg; b < b_end; ++b) {
        const Brick k = brick_at(b);
        __syncthreads();  // every wave is done reading the previous brick
        commit();
        __syncthreads();
        if (b + 1 < b_end) fetch(brick_at(b + 1));
        // K step s covers rows (h0 + 2*(s%4) + {0,1}) of depth d0 + s/4; dy
        // rows for step s+1 are fetched while step s multiplies
        auto load_a = [&](int s, F16B (&av)[4]) {
            const int dl = s / (kWH / 2);
            const int hl = (s % (kWH / 2)) * 2 + hl_l;
            const int d = k.d0 + dl, h = k.h0 + hl, w = k.w0 + wl;
            const bool ok = d < a.D && h < a.H && w + 8 <= a.W;
#pragma unroll
            for (int ct = 0; ct < 4; ++ct) {
                av[ct].u = make_uint4(0u, 0u, 0u, 0u);
                if (ok)
                    av[ct].u = *reinterpret_cast<const uint4*>(
                        a.dy + ((int64_t)k.n * a.Co + co0 + ct * 16 + li) * V + d * HW +
                        (int64_t)h * a.W + w);
            }
        };
        F16B ac[4];
        load_a(0, ac);
#pragma unroll 1
        for (int s = 0; s < kWD * kWH / 2; ++s) {
            F16B an[4];
            load_a(s + 1 < kWD * kWH / 2 ? s + 1 : s, an);
            const int dl = s / (kWH / 2);
            const int hl = (s % (kWH / 2)) * 2 + hl_l;
#pragma unroll
            for (int j = 0; j < NTAP; ++j) {
                const int t = wave + 4 * j;
                if (t < KT) {
                    const int kd = t / (KS * KS), kh = (t / KS) % KS, kw = t % KS;
                    F16B bv;
                    bv.u = *reinterpret_cast<const uint4*>(
                        xs + kw * KWS + li * CIS + ((dl + kd) * PH + hl + kh) * 32 + wl * 2);
#pragma unroll
                    for (int ct = 0; ct < 4; ++ct) acc[j][ct] = mfma(ac[ct], bv, acc[j][ct]);
                }
            }
#pragma unroll
            for (int ct = 0; ct < 4; ++ct) ac[ct] = an[ct];
        }
    }

    float* out = a.part + (int64_t)L * kWgPart + tid;
#pragma unroll
    for (int j = 0; j < NTAP; ++j)
#pragma unroll
        for (int ct = 0; ct < 4; ++ct)
#pragma unroll
            for (int e = 0; e < 4; ++e) out[((j * 4 + ct) * 4 + e) * 256] = acc[j][ct][e];
}

// dw[co][ci][t] (+)= sum over ranges, in range order, of the partial element
// that holds (co, ci, t).  One thread per partial element of a workgroup
// tile (group = cig + cigs * cog), reading the ranges with coalesced loads.
__global__ __launch_bounds__(256) void wgrad_brick_reduce(const float* __restrict__ part,
                                                          int ranges, int groups, int cigs,
                                                          int Ci, float* __restrict__ dw,
                                                          int accumulate) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (int64_t)groups * kWgPart) return;
    const int group = (int)(i / kWgPart), r = (int)(i - (int64_t)group * kWgPart);
    const int tid = r & 255, jce = r >> 8;
    const int e = jce & 3, ct = (jce >> 2) & 3, j = jce >> 4;
    const int wave = tid >> 6, lane = tid & 63;
    const int t = wave + 4 * j;
    if (t >= 27) return;
    const int cig = group % cigs, cog = group / cigs;
    const int co = cog * 64 + ct * 16 + 4 * (lane >> 4) + e;
    const int ci = cig * 16 + (lane & 15);
    const int64_t stride = (int64_t)groups * kWgPart;
    float s = 0.f;
#pragma unroll 8
    for (int z = 0; z < ranges; ++z) s += part[(int64_t)z * stride + i];
    float* o = dw + ((int64_t)co * Ci + ci) * 27 + t;
    *o = accumulate ? *o + s : s;
}

// ---------------------------------------------------------------- dispatch
bool brick_fd_ok(const ConvGeom& g, rat3d_dtype dt, bool dgrad) {
    if (dt != RAT3D_BF16 || g.s != 1) return false;
    if (!((g.k == 3 && g.p == 1) || (g.k == 1 && g.p == 0))) return false;
    const int cs = dgrad ? g.Co : g.Ci, ct = dgrad ? g.Ci : g.Co;
    return cs % 32 == 0 && ct % 32 == 0;
}

bool brick_wgrad_ok(const ConvGeom& g, rat3d_dtype dt) {
    return dt == RAT3D_BF16 && g.s == 1 && g.k == 3 && g.p == 1 && g.Ci % 16 == 0 &&
           g.Co % 64 == 0 && g.W % 8 == 0;
}

size_t brick_fd_ws(const ConvGeom& g) { return (size_t)g.Co * g.Ci * g.k * g.k * g.k * 2; }

static int wgrad_ranges(const ConvGeom& g, int64_t nbricks) {
    // about two workgroups per CU in one wave (256 CUs, 2 resident each)
    const int64_t groups = (int64_t)(g.Ci / 16) * (g.Co / 64);
    int64_t r = ceil_div(512, groups);
    if (r > nbricks) r = nbricks;
    if (r < 1) r = 1;
    return (int)r;
}

static int64_t wgrad_bricks(const ConvGeom& g) {
    return (int64_t)g.N * ceil_div(g.D, kWD) * ceil_div(g.H, kWH) * ceil_div(g.W, kWW);
}

size_t brick_wgrad_ws(const ConvGeom& g) {
    const int R = wgrad_ranges(g, wgrad_bricks(g));
    return (size_t)R * (g.Ci / 16) * (g.Co / 64) * kWgPart * sizeof(float);
}

rat3d_status conv_fd_brick(const ConvGeom& g, bool dgrad, const void* src, const void* w,
                           const float* bias, void* dst, int accumulate, void* ws,
                           hipStream_t st) {
    const int KT = g.k * g.k * g.k;
    bf16* wt = (bf16*)ws;
    const int64_t wn = (int64_t)g.Co * g.Ci * KT;
    if (dgrad)
        prep_dgrad_weights<<<(unsigned)ceil_div(wn, 256), 256, 0, st>>>((const bf16*)w, g.Co,
                                                                        g.Ci, KT, wt);
    else
        prep_fwd_weights<<<(unsigned)ceil_div(wn, 256), 256, 0, st>>>((const bf16*)w, g.Co, g.Ci,
                                                                      KT, wt);
    RAT3D_LAUNCH_CHECK();
    FdArgs a;
    a.src = (const bf16*)src;
    a.wt = wt;
    a.bias = bias;
    a.dst = (bf16*)dst;
    a.N = g.N;
    a.Cs = dgrad ? g.Co : g.Ci;
    a.Ct = dgrad ? g.Ci : g.Co;
    a.D = g.D;
    a.H = g.H;
    a.W = g.W;
    a.td = (int)ceil_div(g.D, kBD);
    a.th = (int)ceil_div(g.H, kBH);
    a.tw = (int)ceil_div(g.W, kBW);
    a.accumulate = accumulate;
    const int nt = a.Ct % 64 == 0 ? 4 : 2;
    dim3 grid((unsigned)((int64_t)g.N * a.td * a.th * a.tw), (unsigned)(a.Ct / (nt * 16)));
    ProfScope ps(dgrad ? (g.k == 3 ? "conv_brick3_dgrad" : "conv_brick1_dgrad")
                       : (g.k == 3 ? "conv_brick3_fwd" : "conv_brick1_fwd"),
                 st, conv_flops(g), conv_bytes(g, 2));
    if (g.k == 3) {
        if (nt == 4) conv_brick_fd<3, 4><<<grid, 256, 0, st>>>(a);
        else conv_brick_fd<3, 2><<<grid, 256, 0, st>>>(a);
    } else {
        if (nt == 4) conv_brick_fd<1, 4><<<grid, 256, 0, st>>>(a);
        else conv_brick_fd<1, 2><<<grid, 256, 0, st>>>(a);
    }
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

rat3d_status conv_wgrad_brick(const ConvGeom& g, const void* x, const void* dy, float* dw,
                              int accumulate, void* ws, hipStream_t st) {
    WgArgs a;
    a.x = (const bf16*)x;
    a.dy = (const bf16*)dy;
    a.part = (float*)ws;
    a.N = g.N;
    a.Ci = g.Ci;
    a.Co = g.Co;
    a.D = g.D;
    a.H = g.H;
    a.W = g.W;
    a.td = (int)ceil_div(g.D, kWD);
    a.th = (int)ceil_div(g.H, kWH);
    a.tw = (int)ceil_div(g.W, kWW);
    a.nbricks = wgrad_bricks(g);
    const int R = wgrad_ranges(g, a.nbricks);
    a.bpr = (int)ceil_div(a.nbricks, R);
    const int Rreal = (int)ceil_div(a.nbricks, a.bpr);
    a.cigs = g.Ci / 16;
    a.cogs = g.Co / 64;
    {
        ProfScope ps("conv_brick3_wgrad", st, conv_flops(g), conv_bytes(g, 2));
        conv_brick_wgrad<3><<<(unsigned)((int64_t)Rreal * a.cigs * a.cogs), 256, 0, st>>>(a);
        RAT3D_LAUNCH_CHECK();
    }
    const int groups = a.cigs * a.cogs;
    const int64_t count = (int64_t)groups * kWgPart;
    ProfScope ps("wgrad_reduce", st, 0.0,
                 4.0 * (count * Rreal + (double)g.Co * g.Ci * 27 * (1 + accumulate)));
    wgrad_brick_reduce<<<(unsigned)ceil_div(count, 256), 256, 0, st>>>(
        a.part, Rreal, groups, a.cigs, g.Ci, dw, accumulate);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

}  // namespace rat3d
