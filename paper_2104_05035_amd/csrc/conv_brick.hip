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
#include <cstdio>

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
constexpr int kWH = 8, kWW = 16;              // weight-gradient voxel brick (one depth slice)

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
    int cogs;          // output-channel groups of NT * 16
    int ntiles;        // work items: N * td * th * tw * cogs * nsplit
    int accumulate;
    // split over the source channels (maps too small to occupy every CU):
    // item = (tile, split) sums chunks [split * cps, (split + 1) * cps) and
    // stores fp32 partials, part[split][n][co][v], summed by brick_split_reduce
    int nsplit, cps;
    float* part;
};

}  // namespace

// ---------------------------------------------------------------- weight prep
// Prepared layouts (source channels innermost, in chunks of 32; Cs is a
// multiple of 32 on every path that reads them):
//   fwd:   wt[((c/32)*KT + t)*Co + co]*32 + c%32] = w[co][c][t]
//   dgrad: wt[((co/32)*KT + t)*Ci + ci]*32 + co%32] = w[co][ci][KT - 1 - t]
// Several convolutions' layouts in one launch: job j covers 16-byte
// destination units [begin_j, begin_j + Co*Ci*KT/8).  One thread per unit
// (eight consecutive source channels): eight gathered 2-byte reads (cached)
// and one 16-byte store, so the writes are whole, contiguous lines.
struct PrepBatch {
    const bf16* w[kPrepJobs];
    bf16* wt[kPrepJobs];
    int co[kPrepJobs], ci[kPrepJobs], kt[kPrepJobs], dg[kPrepJobs];
    int64_t begin[kPrepJobs + 1];
    int n;
};

__global__ void prep_weights_batch(PrepBatch b) {
    const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (u >= b.begin[b.n]) return;
    int lo = 0, hi = b.n - 1;  // the job whose range holds u
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (b.begin[mid] <= u) lo = mid;
        else hi = mid - 1;
    }
    const int64_t e = u - b.begin[lo];
    const int KT = b.kt[lo], Ci = b.ci[lo], Co = b.co[lo];
    const bool dg = b.dg[lo] != 0;
    const int Ct = dg ? Ci : Co;  // target channels (the row index of the layout)
    // e = ((cb * KT + t) * Ct + tc) * 4 + s8: unit s8 of the 32 source channels of chunk cb
    const int s8 = (int)(e & 3);
    const int64_t r = e >> 2;
    const int tc = (int)(r % Ct);
    const int64_t r2 = r / Ct;
    const int t = (int)(r2 % KT), cb = (int)(r2 / KT);
    const int s0 = cb * 32 + s8 * 8;
    const bf16* w = b.w[lo];
    // fwd: w[tc][s][t]; dgrad: w[s][tc][KT - 1 - t]
    const int64_t base = dg ? ((int64_t)s0 * Ci + tc) * KT + (KT - 1 - t)
                            : ((int64_t)tc * Ci + s0) * KT + t;
    const int64_t step = dg ? (int64_t)Ci * KT : KT;
    uint32_t v[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) v[j] = w[base + j * step];
    *reinterpret_cast<uint4*>(b.wt[lo] + e * 8) =
        make_uint4(v[0] | (v[1] << 16), v[2] | (v[3] << 16), v[4] | (v[5] << 16),
                   v[6] | (v[7] << 16));
}

rat3d_status brick_prep_weights_batch(const PrepJob* jobs, int n, hipStream_t st) {
    for (int j = 0; j < n; ++j) {
        const int cs = jobs[j].dgrad ? jobs[j].g.Co : jobs[j].g.Ci;
        if (cs % 32 != 0 || ((uintptr_t)jobs[j].wt & 15u)) {
            set_error("weight layout: source channels (%d) must be a multiple of 32 and the "
                      "prepared buffer 16-byte aligned", cs);
            return RAT3D_EINVAL;
        }
    }
    for (int j0 = 0; j0 < n; j0 += kPrepJobs) {
        PrepBatch b{};
        b.n = n - j0 < kPrepJobs ? n - j0 : kPrepJobs;
        b.begin[0] = 0;
        for (int j = 0; j < b.n; ++j) {
            const PrepJob& J = jobs[j0 + j];
            b.w[j] = (const bf16*)J.w;
            b.wt[j] = (bf16*)J.wt;
            b.co[j] = J.g.Co;
            b.ci[j] = J.g.Ci;
            b.kt[j] = J.g.k * J.g.k * J.g.k;
            b.dg[j] = J.dgrad ? 1 : 0;
            b.begin[j + 1] = b.begin[j] + (int64_t)J.g.Co * J.g.Ci * b.kt[j] / 8;
        }
        prep_weights_batch<<<(unsigned)ceil_div(b.begin[b.n], 256), 256, 0, st>>>(b);
        RAT3D_LAUNCH_CHECK();
    }
    return RAT3D_OK;
}

// ---------------------------------------------------------------- fwd / dgrad
// LDS brick layout: voxel v = (dd * PH + hh) * PW + ww holds 64 bytes, four
// 16-byte slots of eight channels; channel group cg sits in slot
// cg ^ ((ww >> 1) & 3).  The swizzle depends on the brick column only, so the
// eight rows a wave reads for one tap differ by constant offsets, and any
// eight consecutive columns (64 bytes apart) get distinct (column parity,
// slot) pairs: distinct 16-byte bank groups of a 128-byte bank row.
__device__ __forceinline__ int brick_swizzle(int ww) { return (ww >> 1) & 3; }
template <int KS>
__device__ __forceinline__ uint32_t brick_slot_off(int ww, int cg) {
    return (uint32_t)(ww * 64 + ((cg ^ brick_swizzle(ww)) << 4));
}

__device__ __forceinline__ uint32_t pack_lo(uint32_t lo, uint32_t hi) {
    return __builtin_amdgcn_perm(hi, lo, 0x05040100u);  // lo16(lo) | lo16(hi) << 16
}
__device__ __forceinline__ uint32_t pack_hi(uint32_t lo, uint32_t hi) {
    return __builtin_amdgcn_perm(hi, lo, 0x07060302u);  // hi16(lo) | hi16(hi) << 16
}

// Persistent producer/consumer kernel, one 512-thread workgroup per CU.
// Waves 0-3 (consumers) multiply: each owns one output depth slice of the
// 4 x 8 x 16 tile, 8 rows x NT*16 channels of accumulators.  Waves 4-7
// (producers) stage the next (tile, 32-channel chunk) step into the other of
// two LDS brick buffers while the consumers work on the current one; a step
// ends with one workgroup barrier.  A workgroup walks its tiles in a fixed
// order: with a grid that is a multiple of 8, the workgroups of one XCD share
// a contiguous range of tiles, so halo lines are reused from that XCD's L2.
// Workgroup barrier that orders LDS accesses only (no wait for global stores).
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int KS, int NT, int RD, bool ACC, bool DG>
__global__ __launch_bounds__(512, 1) void conv_brick_fd(FdArgs a) {
    constexpr int P = (KS - 1) / 2;
    constexpr int PD = kBD + KS - 1, PH = kBH + KS - 1, PW = kBW + KS - 1;
    constexpr int NV = PD * PH * PW;
    constexpr int KT = KS * KS * KS;
    // Brick row stride, padded to an odd multiple of 32 bytes.  Measured on
    // gfx950 with 16-byte LDS accesses whose 16-lane groups step through rows
    // of stride S: S = 32 or 96 (mod 128) is conflict-free, S = 16, 48, 80 or
    // 112 (mod 128) costs two passes, S = 0 (mod 128) four or more.  A bare row
    // of 18 or 16 voxels x 64 bytes is a multiple of 128 bytes, so without the
    // padding the lanes of one staging store (the same column of different
    // rows) would all hit the same banks.
    constexpr uint32_t RS = PW * 64 + 32;
    constexpr uint32_t BB = PD * PH * RS;       // bytes per brick buffer
    // 1^3: the output tile does not fit a brick buffer and gets its own region
    // (co stride padded to an odd multiple of 32 bytes, as the row stride)
    constexpr uint32_t OCS = kBD * kBH * kBW * 2 + 32;
    constexpr uint32_t OB = KS == 1 ? NT * 16 * OCS : 0;
    __shared__ __align__(16) unsigned char lds[2 * BB + OB];

    // wave index made explicitly uniform: values derived from it (weight offsets)
    // then stay in scalar registers instead of forcing per-lane loops
    const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
    const bool consumer = wave < 4;
    const int HW = a.H * a.W, V = HW * a.D;
    const uint32_t Vb = (uint32_t)V * 2u;

    int t_first, t_stride, t_end;
    {
        const int G = gridDim.x, b = blockIdx.x;
        if ((G & 7) == 0) {
            const int x = b & 7;
            t_first = (int)((int64_t)a.ntiles * x / 8) + (b >> 3);
            t_stride = G >> 3;
            t_end = (int)((int64_t)a.ntiles * (x + 1) / 8);
        } else {
            t_first = b;
            t_stride = G;
            t_end = a.ntiles;
        }
    }
    const int S = (t_first < t_end ? (t_end - t_first + t_stride - 1) / t_stride : 0) * a.cps;

    struct Tile {
        int n, d0, h0, w0, co0, split;
    };
    auto tile_of = [&](int k) {
        int r = t_first + (k / a.cps) * t_stride;
        Tile T;
        T.split = r % a.nsplit;
        r /= a.nsplit;
        T.co0 = (r % a.cogs) * NT * 16;
        r /= a.cogs;
        T.w0 = (r % a.tw) * kBW;
        r /= a.tw;
        T.h0 = (r % a.th) * kBH;
        r /= a.th;
        T.d0 = (r % a.td) * kBD;
        T.n = r / a.td;
        return T;
    };

    // ---- producer.  Staging item = (channel group cg, brick row, 8-column
    // group q): eight 16-byte loads (one per channel) of 8 consecutive input
    // columns, transposed in registers into 8 voxels x 8 channels.  q runs
    // fastest, so the lanes of one load read adjacent 16-byte pieces of a row.
    // Groups start at w0 - 8 (3^3: only its last column is the left halo) and
    // end at w0 + 23 (3^3: only w0 + 16 is used).
    constexpr int Q0 = KS == 3 ? -1 : 0;       // first group, in 8-column units from w0
    constexpr int NQ = KS == 3 ? 4 : 2;        // groups per brick row
    constexpr int NPAIR = 4 * PD * PH;         // (channel group, brick row) pairs
    constexpr int NIT = NPAIR * NQ;            // staging items per step
    constexpr int NRND = (NIT + 255) / 256;    // items per producer thread
    static_assert(NPAIR * PW >= NT * 16 * kBD * kBH * 2 || KS != 3, "epilogue slots");
    const int ptid = tid - 256;
    auto item_of = [&](int r, int& pair, int& q) {
        const int it = ptid + 256 * r;
        pair = it / NQ;
        q = it - pair * NQ;
        return it < NIT;
    };
    // Aligned widths: stage_load issues the loads of a block of the step's
    // items (registers v, items i0 ..), stage_write transposes them into the
    // buffer.  The producer stages in blocks of two items after it has
    // drained the previous tile's outputs (issuing all loads before the drain
    // measured slower).
    // first source channel of step k's 32-channel chunk
    auto chunk_c0 = [&](const Tile& T, int k) { return (T.split * a.cps + k % a.cps) * 32; };
    auto stage_load = [&](int k, auto& v, int i0) {
        constexpr int NB = sizeof(v) / sizeof(v[0]);
        const Tile T = tile_of(k);
        const int c0 = chunk_c0(T, k);
        const __amdgpu_buffer_rsrc_t src_r =
            buf_rsrc_u(a.src + (int64_t)T.n * a.Cs * V, (uint32_t)a.Cs * Vb);
#pragma unroll
        for (int ii = 0; ii < NB; ++ii) {
            int pair, q;
            const bool live = i0 + ii < NRND && item_of(i0 + ii, pair, q);
            const int cg = pair / (PD * PH), row = pair - cg * (PD * PH);
            const int dd = row / PH, hh = row - dd * PH;
            const int d = T.d0 - P + dd, h = T.h0 - P + hh, wg = T.w0 + 8 * (q + Q0);
            const bool ok = live && (unsigned)d < (unsigned)a.D && (unsigned)h < (unsigned)a.H &&
                            (unsigned)wg < (unsigned)a.W;
            // an offset past the buffer end reads zeros (padding)
            const uint32_t vo = ok ? (uint32_t)((cg * 8 * V + d * HW + h * a.W + wg) * 2) : 0x80000000u;
#pragma unroll
            for (int j = 0; j < 8; ++j) v[ii][j] = buf_ld16(src_r, vo, (uint32_t)(c0 + j) * Vb);
        }
    };
    auto stage_write = [&](unsigned char* buf, const auto& v, int i0) {
        constexpr int NB = sizeof(v) / sizeof(v[0]);
#pragma unroll
        for (int ii = 0; ii < NB; ++ii) {
            int pair, q;
            if (!(i0 + ii < NRND && item_of(i0 + ii, pair, q))) continue;
            const int cg = pair / (PD * PH), row = pair - cg * (PD * PH);
            unsigned char* rb = buf + (uint32_t)row * RS;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int ww = 8 * (q + Q0) + e + P;  // brick column
                if (ww < 0 || ww >= PW) continue;
                const int wd = e >> 1;
                uint32_t o[4];
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    const uint32_t wl = wd == 0 ? v[ii][2 * c].x
                                      : wd == 1 ? v[ii][2 * c].y
                                      : wd == 2 ? v[ii][2 * c].z : v[ii][2 * c].w;
                    const uint32_t wh = wd == 0 ? v[ii][2 * c + 1].x
                                      : wd == 1 ? v[ii][2 * c + 1].y
                                      : wd == 2 ? v[ii][2 * c + 1].z : v[ii][2 * c + 1].w;
                    o[c] = (e & 1) ? pack_hi(wl, wh) : pack_lo(wl, wh);
                }
                *reinterpret_cast<uint4*>(rb + brick_slot_off<KS>(ww, cg)) =
                    make_uint4(o[0], o[1], o[2], o[3]);
            }
        }
    };
    // Widths that are not a multiple of 8: item = (channel group, brick
    // voxel), voxel fastest, loaded and written in one pass.
    auto stage_generic = [&](int k, unsigned char* buf) {
        const Tile T = tile_of(k);
        const int c0 = chunk_c0(T, k);
        {
            // item = (channel group, brick voxel), voxel fastest
            for (int it = ptid; it < NV * 4; it += 256) {
                const int vox = it % NV, cg = it / NV;
                const int ww = vox % PW, rr = vox / PW;
                const int hh = rr % PH, dd = rr / PH;
                const int d = T.d0 - P + dd, h = T.h0 - P + hh, w = T.w0 - P + ww;
                uint4 pk = make_uint4(0u, 0u, 0u, 0u);
                if ((unsigned)d < (unsigned)a.D && (unsigned)h < (unsigned)a.H &&
                    (unsigned)w < (unsigned)a.W) {
                    const bf16* p = a.src + ((int64_t)T.n * a.Cs + c0 + cg * 8) * V +
                                    (int64_t)d * HW + (int64_t)h * a.W + w;
                    uint32_t u[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) u[j] = p[(int64_t)j * V];
                    pk.x = u[0] | (u[1] << 16);
                    pk.y = u[2] | (u[3] << 16);
                    pk.z = u[4] | (u[5] << 16);
                    pk.w = u[6] | (u[7] << 16);
                }
                *reinterpret_cast<uint4*>(buf + (uint32_t)rr * RS +
                                          brick_slot_off<KS>(ww, cg)) = pk;
            }
        }
    };

    // ---- consumer.  The four consumer waves split the tile as WD depth groups
    // (RD slices of 8 rows each) x WC output-channel groups (CT x 16
    // channels); lane (li, kg) reads brick column li + kw, channel slot kg.
    constexpr int WD = kBD / RD, WC = 4 / WD, CT = NT / WC, NR = RD * kBH;
    static_assert(WD * RD == kBD && WC * WD == 4 && CT * WC == NT, "wave split");
    const int li = lane & 15, kg = lane >> 4;
    const int wd = (wave & 3) % WD, wc = (wave & 3) / WD;
    uint32_t sw[KS];
#pragma unroll
    for (int kw = 0; kw < KS; ++kw)
        sw[kw] = (uint32_t)(wd * RD * PH) * RS + brick_slot_off<KS>(li + kw, kg);
    const uint32_t wlane = (uint32_t)(li * 64 + kg * 16);
    const __amdgpu_buffer_rsrc_t wt_r =
        buf_rsrc(a.wt, (uint32_t)(a.Cs / 32) * KT * (uint32_t)a.Ct * 64u);
    f32x4 acc[NR][CT];
    // brick offset of the wave's row r (depth slice r / 8, tile row r % 8)
    auto row_off = [](int r) { return ((r / kBH) * PH + (r % kBH)) * (int)RS; };

    auto compute = [&](int k, const unsigned char* buf) {
        const Tile T = tile_of(k);
        const int c0 = chunk_c0(T, k);
        if (k % a.cps == 0) {
#pragma unroll
            for (int i = 0; i < NR; ++i)
#pragma unroll
                for (int j = 0; j < CT; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
        }
        // weight fragments [chunk][tap][Ct][32].  B operands of tap t+1 are
        // fetched while tap t multiplies.  A operands stream through a ring of
        // LA registers: operand g = tap * NR + row is read LA rows ahead of its
        // MFMAs, into the slot the MFMAs of operand g have just released.
        constexpr int LA = NR < 10 ? NR : 10;
        constexpr int NG = KT * NR;
        const uint32_t wchunk =
            ((uint32_t)(c0 >> 5) * KT * (uint32_t)a.Ct + T.co0 + wc * CT * 16) * 64u;
        constexpr int LB = 2;  // weight taps loaded ahead of the current one
        F16B A[LA], B[LB + 1][CT];
        auto a_ptr = [&](int g) {
            const int tap = g / NR, r = g % NR;
            const int kd = tap / (KS * KS), kh = (tap / KS) % KS, kw = tap % KS;
            return buf + sw[kw] + (kd * PH + kh) * (int)RS + row_off(r);
        };
        auto load_b = [&](int tap, F16B (&bv)[CT]) {
#pragma unroll
            for (int ct = 0; ct < CT; ++ct)
                bv[ct].u = buf_ld16(wt_r, wlane, wchunk + ((uint32_t)tap * a.Ct + ct * 16) * 64u);
        };
#pragma unroll
        for (int g = 0; g < LA; ++g) A[g].u = *reinterpret_cast<const uint4*>(a_ptr(g));
#pragma unroll
        for (int tap = 0; tap < LB && tap < KT; ++tap) load_b(tap, B[tap]);
#pragma unroll
        for (int tap = 0; tap < KT; ++tap) {
            if (tap + LB < KT) load_b(tap + LB, B[(tap + LB) % (LB + 1)]);
#pragma unroll
            for (int r = 0; r < NR; ++r) {
                const int g = tap * NR + r;
#pragma unroll
                for (int ct = 0; ct < CT; ++ct)
                    acc[r][ct] = mfma(A[g % LA], B[tap % (LB + 1)][ct], acc[r][ct]);
                if (g + LA < NG) A[g % LA].u = *reinterpret_cast<const uint4*>(a_ptr(g + LA));
            }
            // issue order within a tap: the next tap's weight loads, then per
            // row its MFMAs followed by the ring refill; nothing moves across
            // taps (register pressure)
            if (tap + LB < KT) {
                __builtin_amdgcn_sched_group_barrier(0x020, CT, 0);
#pragma unroll
                for (int r = 0; r < NR; ++r) {
                    __builtin_amdgcn_sched_group_barrier(0x008, CT, 0);
                    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // Output epilogue, staged: after a tile's last MFMA the consumers write
    // bf16 results (bias added) into the brick buffer they just finished
    // reading, in 16-byte units of eight w.  Channel group cg (16 channels)
    // uses channel slot cg; its output rows rho = (d * 8 + h) * 16 + co % 16
    // (16 w = two units each) are placed so that the producer lanes of one
    // store instruction hold both units of a row, which makes every global
    // store cover whole 32-byte row pieces:
    //   rho < 480        units in brick row rho / 8, columns rho % 8 + 1 and
    //                    rho % 8 + 9 (the column groups of staging items q = 1
    //                    and q = 2 of one brick row, same column offset);
    //   rho = 480 + j    column 0 of brick rows 2j and 2j + 1 (j < 30), or
    //                    column 17 of brick rows 2(j - 30) and 2(j - 30) + 1.
    // Each unit sits in a slot that one staging item writes; the producer
    // thread that owns the item stores the unit to global memory before it
    // stages into the buffer again, so no producer overwrites a unit another
    // has not drained, and the global stores (and any wait for them) stay off
    // the consumer waves.
    auto dst_rsrc = [&](const Tile& T) {
        return buf_rsrc_u(a.dst + (int64_t)T.n * a.Ct * V, (uint32_t)a.Ct * Vb);
    };
    constexpr int kRowsMain = PD * PH * 8;  // rows in columns 1 .. 16
    static_assert(KS != 3 || (PW == 18 && kRowsMain + PD * PH / 2 + 2 >= 16 * kBD * kBH),
                  "staged outputs fit the brick");
    // Accumulating 3^3 outputs take the same path: the consumer lanes load
    // the old values of the results they hold (all loads of a tile in flight
    // together, after the tile's last MFMA has freed the operand registers)
    // and add them before the single rounding; the producers' stores stay
    // plain bf16 stores.
    const bool split_out = a.nsplit > 1;
    const bool staged_epi = !split_out && (!ACC || KS == 3) && (a.W & 7) == 0;
    using OldV = uint2[ACC ? NR : 1][ACC ? CT : 1];
    auto load_old = [&](int k, OldV& o) {
        const Tile T = tile_of(k);
        const __amdgpu_buffer_rsrc_t dst_r = dst_rsrc(T);
        const int w = T.w0 + 4 * kg;
        // lanes past the width read zeros (offset past the buffer end); the
        // producers never store those units
        const uint32_t lo =
            w < a.W ? (uint32_t)(((T.co0 + wc * CT * 16 + li) * V + w) * 2) : 0x80000000u;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const int d = T.d0 + wd * RD + r / kBH, h = T.h0 + r % kBH;  // wave-uniform
            const bool ok = d < a.D && h < a.H;
            const uint32_t so = ok ? (uint32_t)((d * HW + h * a.W) * 2) : 0u;
#pragma unroll
            for (int ct = 0; ct < CT; ++ct)
                o[r][ct] = ok ? buf_ld8(dst_r, lo + (uint32_t)(ct * 16 * V * 2), so)
                              : make_uint2(0u, 0u);
        }
    };
    auto write_outputs = [&](int k, unsigned char* buf, const OldV& old) {
        const Tile T = tile_of(k);
        float bv[CT];
#pragma unroll
        for (int ct = 0; ct < CT; ++ct)
            bv[ct] = !DG && a.bias ? a.bias[T.co0 + (wc * CT + ct) * 16 + li] : 0.f;
        if constexpr (KS == 1) {
            // separate region: unit (co, d, h, half) at co * OCS + ((d * 8 + h) * 2 + half) * 16
            unsigned char* ob = lds + 2 * BB;
            int lane_o = (int)((uint32_t)((wc * CT) * 16 + li) * OCS) +
                         ((wd * RD * kBH) * 2 + (kg >> 1)) * 16 + (kg & 1) * 8;
            asm volatile("" : "+v"(lane_o));
#pragma unroll
            for (int r = 0; r < NR; ++r) {
#pragma unroll
                for (int ct = 0; ct < CT; ++ct)
                    *reinterpret_cast<uint2*>(ob + lane_o + ct * 16 * OCS + r * 32) = make_uint2(
                        pack_bf16x2(acc[r][ct][0] + bv[ct], acc[r][ct][1] + bv[ct]),
                        pack_bf16x2(acc[r][ct][2] + bv[ct], acc[r][ct][3] + bv[ct]));
                __builtin_amdgcn_sched_barrier(0);
            }
            return;
        }
        // opaque per call: keeps the slot arithmetic from being hoisted out of
        // the step loop, where its results would stay live (register pressure)
        int lane_r = li;
        asm volatile("" : "+v"(lane_r));
        const int half = kg >> 1;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const int dh = (wd * RD + r / kBH) * kBH + r % kBH;  // wave-uniform
            const int rho = dh * 16 + lane_r;
            int row, col;
            if (dh * 16 < kRowsMain) {
                row = rho >> 3;
                col = (rho & 7) + 1 + 8 * half;
            } else {
                const int j = rho - kRowsMain;
                const bool c0 = j < PD * PH / 2;
                row = (c0 ? 2 * j : 2 * (j - PD * PH / 2)) + half;
                col = c0 ? 0 : PW - 1;
            }
            unsigned char* base = buf + (uint32_t)row * RS + (uint32_t)col * 64u + (kg & 1) * 8;
            const int sk = brick_swizzle(col);
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                float v0 = acc[r][ct][0] + bv[ct], v1 = acc[r][ct][1] + bv[ct];
                float v2 = acc[r][ct][2] + bv[ct], v3 = acc[r][ct][3] + bv[ct];
                if constexpr (ACC) {
                    const uint2 o = old[r][ct];
                    v0 += __uint_as_float(o.x << 16);
                    v1 += __uint_as_float(o.x & 0xffff0000u);
                    v2 += __uint_as_float(o.y << 16);
                    v3 += __uint_as_float(o.y & 0xffff0000u);
                }
                *reinterpret_cast<uint2*>(base + (((wc * CT + ct) ^ sk) << 4)) =
                    make_uint2(pack_bf16x2(v0, v1), pack_bf16x2(v2, v3));
            }
            __builtin_amdgcn_sched_barrier(0);  // one row at a time (register pressure)
        }
    };
    // The units of staging item r: LDS offsets read into v, global byte
    // offsets (within sample T.n) into go; units outside the tile's valid
    // range get go = 0x80000000 and are not stored.  The eight LDS reads of an
    // item are issued together.
    auto unit_read = [&](const Tile& T, const unsigned char* buf, int r, uint4 (&v)[8],
                         uint32_t (&go)[8]) {
        int pair, q;
        const bool live = item_of(r, pair, q);
        const int cg = pair / (PD * PH), row = pair - cg * (PD * PH);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int col = 8 * (q + Q0) + e + P;
            int rho, half;
            if (col == 0) {
                rho = kRowsMain + (row >> 1);
                half = row & 1;
            } else if (col == PW - 1) {
                rho = kRowsMain + PD * PH / 2 + (row >> 1);
                half = row & 1;
            } else {
                rho = row * 8 + ((col - 1) & 7);
                half = col > 8;
            }
            const int li_o = rho & 15, h = (rho >> 4) & (kBH - 1), d = rho >> 7;
            const int dd = T.d0 + d, hh = T.h0 + h, w = T.w0 + 8 * half;
            const bool ok = live && cg < NT && col >= 0 && col < PW &&
                            !(col == PW - 1 && row >= 4) && dd < a.D && hh < a.H && w < a.W;
            go[e] = ok ? (uint32_t)(((T.co0 + cg * 16 + li_o) * V + dd * HW + hh * a.W + w) * 2)
                       : 0x80000000u;
            const uint32_t lo = ok ? (uint32_t)row * RS + brick_slot_off<KS>(col, cg) : 0u;
            v[e] = *reinterpret_cast<const uint4*>(buf + lo);
        }
    };
    auto unit_store = [&](__amdgpu_buffer_rsrc_t dst_r, const uint4 (&v)[8], const uint32_t (&go)[8]) {
#pragma unroll
        for (int e = 0; e < 8; ++e)
            if (go[e] != 0x80000000u) buf_st16(dst_r, v[e], go[e], 0u);
    };
    auto drain_items = [&](const Tile& T, const unsigned char* buf, int r0, int r1) {
        const __amdgpu_buffer_rsrc_t dst_r = dst_rsrc(T);
#pragma unroll 1
        for (int r = r0; r < r1; ++r) {
            uint4 v[8];
            uint32_t go[8];
            unit_read(T, buf, r, v, go);
            unit_store(dst_r, v, go);
        }
    };
    auto drain = [&](int k, const unsigned char* buf) {
        const Tile T = tile_of(k);
        if constexpr (KS == 1) {
            const unsigned char* ob = lds + 2 * BB;
#pragma unroll 4
            for (int u = ptid; u < NT * 16 * kBD * kBH * 2; u += 256) {
                const int co = u >> 6, rest = u & 63;
                const int half = rest & 1, h = (rest >> 1) & (kBH - 1), d = rest >> 4;
                const uint4 v = *reinterpret_cast<const uint4*>(ob + co * OCS + rest * 16);
                const int dd = T.d0 + d, hh = T.h0 + h, w = T.w0 + 8 * half;
                if (dd < a.D && hh < a.H && w < a.W)
                    *reinterpret_cast<uint4*>(a.dst + ((int64_t)T.n * a.Ct + T.co0 + co) * V +
                                              (int64_t)dd * HW + (int64_t)hh * a.W + w) = v;
            }
            return;
        }
        drain_items(T, buf, 0, NRND);
    };
    // split items: fp32 partial sums straight from the accumulators (bias and
    // old values are added by the reduction)
    auto split_outputs = [&](int k) {
        const Tile T = tile_of(k);
        float* pb = a.part + ((int64_t)T.split * a.N + T.n) * a.Ct * (int64_t)V;
        const int w = T.w0 + 4 * kg;
        const bool vec = (a.W & 3) == 0 && w + 4 <= a.W;
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const int d = T.d0 + wd * RD + r / kBH, h = T.h0 + r % kBH;
            if (d >= a.D || h >= a.H) continue;
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                const int co = T.co0 + (wc * CT + ct) * 16 + li;
                float* q = pb + (int64_t)co * V + (int64_t)d * HW + (int64_t)h * a.W + w;
                if (vec) {
                    *reinterpret_cast<float4*>(q) =
                        make_float4(acc[r][ct][0], acc[r][ct][1], acc[r][ct][2], acc[r][ct][3]);
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (w + e < a.W) q[e] = acc[r][ct][e];
                }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // direct epilogue (widths not a multiple of 8, accumulating 1^3):
    // lane holds 4 consecutive w of one output channel per tile row
    auto direct_outputs = [&](int k) {
        const Tile T = tile_of(k);
        const bool full_w = (T.w0 + kBW <= a.W) && ((a.W & 3) == 0);
#pragma unroll
        for (int r = 0; r < NR; ++r) {
            const int d = T.d0 + wd * RD + r / kBH, h = T.h0 + r % kBH;
            if (d >= a.D || h >= a.H) continue;
#pragma unroll
            for (int ct = 0; ct < CT; ++ct) {
                const int co = T.co0 + (wc * CT + ct) * 16 + li;
                const float bv = !DG && a.bias ? a.bias[co] : 0.f;
                const int w = T.w0 + 4 * kg;
                bf16* q = a.dst + ((int64_t)T.n * a.Ct + co) * V + (int64_t)d * HW +
                          (int64_t)h * a.W + w;
                float v[4];
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = acc[r][ct][e] + bv;
                if (full_w) {
                    uint2* q2 = reinterpret_cast<uint2*>(q);
                    if (a.accumulate) {
                        const uint2 o = *q2;
                        v[0] += __uint_as_float(o.x << 16);
                        v[1] += __uint_as_float(o.x & 0xffff0000u);
                        v[2] += __uint_as_float(o.y << 16);
                        v[3] += __uint_as_float(o.y & 0xffff0000u);
                    }
                    *q2 = make_uint2(pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]));
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
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    // Both roles pass the same barriers (one per step, two on a tile's last
    // step with the staged epilogue); the roles are wave-uniform, and the two
    // loops keep the consumers' accumulators out of the producers' live range.
    // The barriers order LDS only: global stores are never waited for.
    auto tile_end = [&](int k) { return (k % a.cps) == a.cps - 1; };
    if (consumer) {
        lds_barrier();
        for (int k = 0; k < S; ++k) {
            unsigned char* buf = lds + (k & 1) * BB;
            compute(k, buf);
            if (tile_end(k) && staged_epi) {
                OldV old;
                if constexpr (ACC) load_old(k, old);
                lds_barrier();  // every consumer is done reading buf
                write_outputs(k, buf, old);
                lds_barrier();
            } else {
                if (tile_end(k)) {
                    if (split_out) split_outputs(k);
                    else direct_outputs(k);
                }
                lds_barrier();
            }
        }
    } else {
        const bool aligned = (a.W & 7) == 0;
        auto stage_all = [&](int k, unsigned char* buf) {
            if (!aligned) {
                stage_generic(k, buf);
                return;
            }
#pragma unroll 1
            for (int i0 = 0; i0 < NRND; i0 += 2) {
                uint4 v[2][8];
                stage_load(k, v, i0);
                stage_write(buf, v, i0);
            }
        };
        // bf16 epilogue of 3^3 tiles: a tile's drain is split over two steps.
        // Items 0 .. NE-1 are stored at once; the units of the other items are
        // read into registers before the buffer is staged again and stored at
        // the start of the next step.  Every workgroup drains at the same
        // steps, so this halves the store burst that meets the next staging.
        constexpr int NE = (NRND + 1) / 2, NL = NRND - NE > 0 ? NRND - NE : 1;
        const bool split = KS == 3 && staged_epi && NRND > 1;
        uint4 late_v[NL][8];
        uint32_t late_go[NL][8];
        int late_k = -1;
        auto late_store = [&]() {
            if (late_k < 0) return;
            const __amdgpu_buffer_rsrc_t dst_r = dst_rsrc(tile_of(late_k));
#pragma unroll
            for (int i = 0; i < NL; ++i) unit_store(dst_r, late_v[i], late_go[i]);
            late_k = -1;
        };
        auto drain_split = [&](int kd, const unsigned char* buf) {
            const Tile T = tile_of(kd);
#pragma unroll
            for (int i = 0; i < NL; ++i) unit_read(T, buf, NE + i, late_v[i], late_go[i]);
            drain_items(T, buf, 0, NE);
            late_k = kd;
        };
        if (S > 0) stage_all(0, lds);
        lds_barrier();
        for (int k = 0; k < S; ++k) {
            const bool more = k + 1 < S;
            if (split) late_store();
            if (k > 0 && tile_end(k - 1)) {
                if (split) {
                    drain_split(k - 1, lds + ((k - 1) & 1) * BB);
                } else if (staged_epi) {
                    drain(k - 1, lds + ((k - 1) & 1) * BB);
                }
            }
            if (more) stage_all(k + 1, lds + ((k + 1) & 1) * BB);
            if (tile_end(k) && staged_epi) {
                lds_barrier();
                lds_barrier();
            } else {
                lds_barrier();
            }
        }
        if (S > 0) {
            if (split) late_store();
            if (staged_epi) {
                drain(S - 1, lds + ((S - 1) & 1) * BB);
            }
        }
    }
}

// ---------------------------------------------------------------- wgrad
namespace {
struct WgArgs {
    const bf16* x;   // [N][Ci][D][H][W]
    const bf16* dy;  // [N][Co][D][H][W]
    float* part;     // [ranges][groups] blocks of kWgPart floats
    int N, Ci, Co, D, H, W;
    int tds, th, tw;  // steps (depth pairs) per column, row tiles, column tiles
    int nsteps;       // N * th * tw * tds
    int spr;          // steps per range
    int cigs, cogs;   // input-channel groups of 16, output-channel groups of 64
};
}  // namespace

// Partials are stored in the accumulators' register order: per workgroup a
// block of kWgPart floats, element ((j * 4 + ct) * 4 + e) * 256 + tid, so every
// store instruction writes 256 contiguous bytes.  wgrad_brick_reduce sums the
// ranges in order and scatters each sum to its (co, ci, tap).
constexpr int kWgNtap = 7;                       // taps per wave: wave + 4 j < 27
constexpr int kWgPart = kWgNtap * 4 * 4 * 256;   // floats per workgroup partial

// Persistent producer/consumer weight gradient, one 512-thread workgroup per
// CU.  A workgroup owns dw for 64 C_out x 16 C_in x 27 taps and sums over a
// range of steps; a step is two 1 x 8 x 16 voxel bricks at depths d0, d0 + 1
// of one (n, row tile, column tile) column, steps ordered depth-fastest.
// Waves 0-3 multiply (wave w owns taps w, w + 4, ...; GEMM K = voxels, A = dy
// rows of 16 output channels, B = x rows of 16 input channels shifted by the
// tap); waves 4-7 stage.  dy of a step goes to one of two LDS buffers; x
// planes live in a ring of six LDS slots (input depth z in slot z mod 6), each
// kept as three kw-shifted copies so that every 8-voxel operand is an aligned
// 16-byte read.  A step needs planes d0 - 1 .. d0 + 2; its successor in the
// same column needs two new planes, whose slots the current step does not
// read, so the producers fill them while the consumers work.  The first step
// of a range or column loads all four planes after the previous step is done
// (one extra barrier).  Producers keep two register sets: the loads for step
// k + 2 are issued during step k and written to LDS during step k + 1.
constexpr int kWgSlots = 6;

template <int KS>
__global__ __launch_bounds__(512, 1) void conv_brick_wgrad(WgArgs a) {
    constexpr int P = (KS - 1) / 2;
    constexpr int KT = KS * KS * KS;
    static_assert(KS == 3, "the weight-gradient brick assembles kw = 0, 1, 2 copies");
    constexpr int PH = kWH + KS - 1;                // x rows per plane
    constexpr int CIS = kWgSlots * PH * 32 + 16;     // bytes per input channel in a copy (+ pad)
    constexpr int KWS = 16 * CIS;                    // bytes per kw-shifted copy
    constexpr int DYS = 2 * kWH * 32 + 16;           // bytes per output channel of a step (+ pad)
    constexpr int DYB = 64 * DYS;                    // bytes per dy buffer
    constexpr int NTAP = (KT + 3) / 4;               // taps per consumer wave
    static_assert(NTAP == kWgNtap, "partial layout");
    constexpr int NXI = (16 * 4 * PH + 255) / 256;   // x staging items per producer thread (full)
    constexpr int NDY = 2 * 64 * kWH * 2 / 256;      // dy staging items (16 bytes) per thread
    __shared__ __align__(16) unsigned char lds[KS * KWS + 2 * DYB];
    unsigned char* const xs = lds;
    unsigned char* const dys = lds + KS * KWS;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const bool consumer = wave < 4;
    const int L = xcd_remap(blockIdx.x, gridDim.x);
    const int groups = a.cigs * a.cogs;
    const int cig = L % a.cigs;
    const int cog = (L / a.cigs) % a.cogs;
    const int range = L / groups;
    const int ci0 = cig * 16, co0 = cog * 64;
    const int s_beg = range * a.spr;
    const int s_end = s_beg + a.spr < a.nsteps ? s_beg + a.spr : a.nsteps;
    const int S = s_end > s_beg ? s_end - s_beg : 0;
    const int64_t HW = (int64_t)a.H * a.W, V = HW * a.D;

    struct Step {
        int n, d0, h0, w0;
        bool full;  // first step of the range or of a column: all four planes
    };
    auto step_at = [&](int k) __attribute__((always_inline)) {
        const int sidx = s_beg + k;
        Step t;
        const int dp = sidx % a.tds;
        int r = sidx / a.tds;
        t.d0 = 2 * dp;
        t.w0 = (r % a.tw) * kWW;
        r /= a.tw;
        t.h0 = (r % a.th) * kWH;
        t.n = r / a.th;
        t.full = k == 0 || dp == 0;
        return t;
    };
    auto slot_of = [](int z) { return (z + kWgSlots) % kWgSlots; };

    // ---- producer
    struct Regs {
        uint32_t m[NXI][10];  // x rows: m[0] = (?, x[w0-1]), m[1..8] = x[w0..w0+15], m[9] = (x[w0+16], ?)
        uint4 dy[NDY];
    };
    const int ptid = tid - 256;
    // x item q of a step: full -> planes d0 - 1 .. d0 + 2, else planes d0 + 1, d0 + 2
    auto x_item = [&](const Step& t, int q, int& ci, int& z, int& row) __attribute__((always_inline)) {
        const int it = ptid + 256 * q;
        const int np = t.full ? 4 : 2;
        ci = it / (np * PH);
        const int rr = it - ci * (np * PH);
        z = (t.full ? t.d0 - P : t.d0 + 1) + rr / PH;
        row = rr % PH;
        return it < 16 * np * PH;
    };
    auto load = [&](const Step& t, Regs& R) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < NXI; ++q) {
#pragma unroll
            for (int j = 0; j < 10; ++j) R.m[q][j] = 0u;
            int ci, z, row;
            if (!x_item(t, q, ci, z, row)) continue;
            const int h = t.h0 - P + row;
            if ((unsigned)z >= (unsigned)a.D || (unsigned)h >= (unsigned)a.H) continue;
            const bf16* p = a.x + ((int64_t)t.n * a.Ci + ci0 + ci) * V + z * HW +
                            (int64_t)h * a.W + t.w0;
            if (t.w0 + 8 <= a.W) {
                const uint4 u = *reinterpret_cast<const uint4*>(p);
                R.m[q][1] = u.x; R.m[q][2] = u.y; R.m[q][3] = u.z; R.m[q][4] = u.w;
            }
            if (t.w0 + 16 <= a.W) {
                const uint4 u = *reinterpret_cast<const uint4*>(p + 8);
                R.m[q][5] = u.x; R.m[q][6] = u.y; R.m[q][7] = u.z; R.m[q][8] = u.w;
            }
            if (t.w0 >= 1) R.m[q][0] = (uint32_t)p[-1] << 16;
            if (t.w0 + 16 < a.W) R.m[q][9] = (uint32_t)p[16];
        }
#pragma unroll
        for (int q = 0; q < NDY; ++q) {
            const int it = ptid + 256 * q;
            const int j = it >> 10, rem = it & 1023;
            const int co = rem >> 4, row = (rem >> 1) & (kWH - 1), half = rem & 1;
            const int d = t.d0 + j, h = t.h0 + row, w = t.w0 + 8 * half;
            R.dy[q] = make_uint4(0u, 0u, 0u, 0u);
            if (d < a.D && h < a.H && w + 8 <= a.W)
                R.dy[q] = *reinterpret_cast<const uint4*>(
                    a.dy + ((int64_t)t.n * a.Co + co0 + co) * V + d * HW + (int64_t)h * a.W + w);
        }
    };
    auto commit_dy = [&](const Regs& R, unsigned char* db) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < NDY; ++q) {
            const int it = ptid + 256 * q;
            const int j = it >> 10, rem = it & 1023;
            const int co = rem >> 4, row = (rem >> 1) & (kWH - 1), half = rem & 1;
            *reinterpret_cast<uint4*>(db + co * DYS + (j * kWH + row) * 32 + half * 16) = R.dy[q];
        }
    };
    // copy kw holds input columns w0 - 1 + kw ... as aligned 16-byte rows
    auto commit_x = [&](const Step& t, const Regs& R) __attribute__((always_inline)) {
#pragma unroll
        for (int q = 0; q < NXI; ++q) {
            int ci, z, row;
            if (!x_item(t, q, ci, z, row)) continue;
            unsigned char* base = xs + ci * CIS + (slot_of(z) * PH + row) * 32;
            const uint32_t* m = R.m[q];
            *reinterpret_cast<uint4*>(base + KWS) = make_uint4(m[1], m[2], m[3], m[4]);
            *reinterpret_cast<uint4*>(base + KWS + 16) = make_uint4(m[5], m[6], m[7], m[8]);
            uint32_t s0[8], s2[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                s0[i] = __builtin_amdgcn_alignbit(m[i + 1], m[i], 16);
                s2[i] = __builtin_amdgcn_alignbit(m[i + 2], m[i + 1], 16);
            }
            *reinterpret_cast<uint4*>(base) = make_uint4(s0[0], s0[1], s0[2], s0[3]);
            *reinterpret_cast<uint4*>(base + 16) = make_uint4(s0[4], s0[5], s0[6], s0[7]);
            *reinterpret_cast<uint4*>(base + 2 * KWS) = make_uint4(s2[0], s2[1], s2[2], s2[3]);
            *reinterpret_cast<uint4*>(base + 2 * KWS + 16) = make_uint4(s2[4], s2[5], s2[6], s2[7]);
        }
    };

    // Barrier schedule (both roles): one prologue barrier, then per step one
    // barrier, plus one more before a step whose x planes are all reloaded.
    if (!consumer) {
        Regs R0, R1;
        if (S > 0) {
            const Step t0 = step_at(0);
            load(t0, R0);
            if (S > 1) load(step_at(1), R1);
            commit_dy(R0, dys);
            commit_x(t0, R0);
        }
        lds_barrier();
        // step k: stage step k + 1 (registers of set (k + 1) & 1), then load
        // step k + 2 into the set just freed; unrolled by two so that the sets
        // are static
        auto body = [&](int k, Regs& Rn, Regs& Rf) __attribute__((always_inline)) {
            // Rn holds step k + 1; Rf is free
            if (k + 1 < S) {
                const Step tn = step_at(k + 1);
                commit_dy(Rn, dys + ((k + 1) & 1) * DYB);
                if (!tn.full) commit_x(tn, Rn);
                if (k + 2 < S) load(step_at(k + 2), Rf);
                lds_barrier();
                if (tn.full) {
                    commit_x(tn, Rn);
                    lds_barrier();
                }
            } else {
                lds_barrier();
            }
        };
        for (int k = 0; k < S; k += 2) {
            body(k, R1, R0);
            if (k + 1 < S) body(k + 1, R0, R1);
        }
        return;
    }

    // ---- consumer
    const int li = lane & 15, kg = lane >> 4;
    const int hl_l = kg >> 1, wl = (kg & 1) * 8;
    f32x4 acc[NTAP][4];
#pragma unroll
    for (int j = 0; j < NTAP; ++j)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[j][c] = f32x4{0.f, 0.f, 0.f, 0.f};

    lds_barrier();
    for (int k = 0; k < S; ++k) {
        const Step t = step_at(k);
        const unsigned char* db = dys + (k & 1) * DYB;
#pragma unroll 1
        for (int j = 0; j < 2; ++j) {
            const int d = t.d0 + j;
            if (d >= a.D) break;
            // plane slot of tap depth kd: input depth d - 1 + kd
            const int sl0 = slot_of(d - 1), sl1 = slot_of(d), sl2 = slot_of(d + 1);
            // K step s covers brick rows 2s, 2s + 1 (32 voxels): lane (li, kg)
            // holds 8 voxels of row 2s + kg/2, columns 8 (kg % 2) ..  The 28
            // operand groups (s, tap slot) run as one straight sequence: the B
            // operand of group g + 3 and, halfway through s, the A operands of
            // s + 1 are read while group g multiplies.  Wave 3's seventh slot
            // repeats tap 26 (kept uniform so the sequence has no branch); its
            // sums are never read.
            const unsigned char* abase = db + li * DYS + (j * kWH + hl_l) * 32 + wl * 2;
            int boff[NTAP];
#pragma unroll
            for (int jj = 0; jj < NTAP; ++jj) {
                int tp = wave + 4 * jj;
                tp = tp < KT ? tp : KT - 1;
                const int kd = tp / (KS * KS), kh = (tp / KS) % KS, kw = tp % KS;
                const int sl = kd == 0 ? sl0 : (kd == 1 ? sl1 : sl2);
                boff[jj] = kw * KWS + li * CIS + (sl * PH + hl_l + kh) * 32 + wl * 2;
            }
            constexpr int G = (kWH / 2) * NTAP;
            constexpr int LA = 3;
            F16B A[2][4], B[4];
#pragma unroll
            for (int ct = 0; ct < 4; ++ct)
                A[0][ct].u = *reinterpret_cast<const uint4*>(abase + ct * 16 * DYS);
#pragma unroll
            for (int g = 0; g < LA; ++g)
                B[g].u = *reinterpret_cast<const uint4*>(xs + boff[g % NTAP] + (g / NTAP) * 64);
#pragma unroll
            for (int g = 0; g < G; ++g) {
                const int s_ = g / NTAP, jj = g % NTAP;
                if (g + LA < G) {
                    const int gn = g + LA;
                    B[gn % 4].u = *reinterpret_cast<const uint4*>(xs + boff[gn % NTAP] +
                                                                  (gn / NTAP) * 64);
                }
                if (jj == 3 && s_ + 1 < kWH / 2) {
#pragma unroll
                    for (int ct = 0; ct < 4; ++ct)
                        A[(s_ + 1) & 1][ct].u = *reinterpret_cast<const uint4*>(
                            abase + ct * 16 * DYS + (s_ + 1) * 64);
                }
#pragma unroll
                for (int ct = 0; ct < 4; ++ct)
                    acc[jj][ct] = mfma(A[s_ & 1][ct], B[g % 4], acc[jj][ct]);
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        lds_barrier();
        if (k + 1 < S && step_at(k + 1).full) lds_barrier();
    }

    float* out = a.part + (int64_t)L * kWgPart + tid;
#pragma unroll
    for (int j = 0; j < NTAP; ++j)
#pragma unroll
        for (int ct = 0; ct < 4; ++ct)
#pragma unroll
            for (int e = 0; e < 4; ++e) out[((j * 4 + ct) * 4 + e) * 256] = acc[j][ct][e];
}

// ---------------------------------------------------------------- band wgrad
// Row-band weight gradient for narrow maps (W a multiple of 4, at most 56).
// A step is one output depth plane d of a band of hb whole rows starting at
// h0, flattened row-major with a row pitch Wp = W rounded up to 8 into the
// GEMM K index (hb * Wp <= NK * 32; pad columns hold dy = 0), so
// every staging load reads whole contiguous rows: the dy of a step is one
// contiguous run of hb * W voxels per output channel and an input plane of
// the band (rows h0 - 1 .. h0 + hb) one contiguous run per input channel.
// Each input plane is kept in LDS as three kw-shifted copies (copy kw holds
// x[h][w + kw - 1], zero where that column is outside the map), so the B
// operand of tap (kd, kh, kw) at flattened voxel v is the aligned 16 bytes at
// v + kh * Wp of copy kw.  The planes of the current step (d - 1, d, d + 1)
// and the next (d + 2) live in a ring of four slots; steps run plane-fastest
// along a band, so a step's producers stage one new plane and the dy of the
// next step while the consumers multiply.  The first step of a range or band
// stages three planes after the previous step is done.  Voxels past hb * W
// in the last K step meet dy = 0 (the LDS is cleared at start).
namespace {
struct WbArgs {
    const bf16* x;   // [N][Ci][D][H][W]
    const bf16* dy;  // [N][Co][D][H][W]
    float* part;     // [ranges][groups] blocks of kWgPart floats
    int N, Ci, Co, D, H, W;
    int Wp, hb, nb;  // LDS row pitch (W rounded up to 8), rows per band, bands per plane
    int nsteps;      // N * nb * D, plane fastest
    int spr;         // steps per range
    int cigs, cogs;  // input-channel groups of 16, output-channel groups of 64
    int sls, cis;    // LDS bytes per plane slot and per input channel (4 slots + pad)
    // ceil(2^20 / divisor) for Wp, the x groups XG = (hb + 2) Wp / 8 of one
    // (channel, plane), 3 XG, and the dy groups YG = hb Wp / 8 of one channel:
    // (i * m) >> 20 == i / divisor for every index the kernel divides
    uint32_t mWp, mXG, m3XG, mYG;
};
constexpr int kBandK = 192;                                  // voxels per step, at most
constexpr int kBandSlotVox = 288;                            // bound on (hb + 2) * W
constexpr int kBandCisMax = 4 * kBandSlotVox * 2 + 32;       // 2336
constexpr int kBandDys = kBandK * 2 + 16;                    // bytes per output channel
constexpr int kBandXBytes = 3 * 16 * kBandCisMax;            // three kw copies
constexpr int kBandLds = kBandXBytes + 2 * 64 * kBandDys;    // 163328
static_assert(kBandLds <= 160 * 1024, "band LDS");
}  // namespace

// MODE: 0 W % 8 = 0 (16-byte loads), 1 W % 8 = 4 (the last group of a row
// holds four voxels: an 8-byte load), 2 any other width (element loads).
template <int NK, int MODE>
__global__ __launch_bounds__(512, 1) void conv_band_wgrad(WbArgs a) {
    constexpr bool PART = MODE == 1, ELEM = MODE == 2;
    constexpr int KT = 27, NTAP = kWgNtap;
    static_assert(NK * 32 <= kBandK, "K steps per band");
    constexpr int DYB = 64 * kBandDys;
    __shared__ __align__(16) unsigned char lds[kBandLds];
    unsigned char* const xs = lds;
    unsigned char* const dys = lds + kBandXBytes;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const bool consumer = wave < 4;
    for (int i = tid; i < kBandLds / 16; i += 512)
        reinterpret_cast<uint4*>(lds)[i] = make_uint4(0u, 0u, 0u, 0u);
    __syncthreads();

    const int L = xcd_remap(blockIdx.x, gridDim.x);
    const int groups = a.cigs * a.cogs;
    const int cig = L % a.cigs;
    const int cog = (L / a.cigs) % a.cogs;
    const int range = L / groups;
    const int ci0 = cig * 16, co0 = cog * 64;
    const int s_beg = range * a.spr;
    const int s_end = s_beg + a.spr < a.nsteps ? s_beg + a.spr : a.nsteps;
    const int S = s_end > s_beg ? s_end - s_beg : 0;
    const int HW = a.H * a.W;
    const int64_t V = (int64_t)HW * a.D;
    const int KWS = 16 * a.cis;

    struct Step {
        int n, d, h0;
        bool full;  // first step of the range or of a band: three planes
    };
    auto step_at = [&](int k) __attribute__((always_inline)) {
        const int sidx = s_beg + k;
        Step t;
        t.d = sidx % a.D;
        const int r = sidx / a.D;
        t.h0 = (r % a.nb) * a.hb;
        t.n = r / a.nb;
        t.full = k == 0 || t.d == 0;
        return t;
    };
    auto slot_of = [](int z) { return (z + 4) & 3; };

    if (!consumer) {
        const int XG = (a.hb + 2) * a.Wp / 8;  // 8-voxel groups of one (channel, plane)
        const int YG = a.hb * a.Wp / 8;        // 8-voxel groups of one output channel
        // PART (W % 8 == 4): the last group of a row holds four voxels (8-byte load)
        auto qdiv = [](int i, uint32_t m) { return (int)(((uint32_t)i * m) >> 20); };
        // The staging index arithmetic is redone at every use (the opaque copy
        // of the thread index keeps it from being hoisted into registers).
        auto ptid_now = [&]() __attribute__((always_inline)) {
            int p = tid - 256;
            asm volatile("" : "+v"(p));
            return p;
        };
        // Staging loads are raw buffer loads over one sample's tensor; an
        // offset past the end (padding, idle item) reads zeros, so no load
        // sits behind a branch.
        // x group: m[0] bits 16..31 = left neighbour, m[1..4] = 8 voxels,
        // m[5] bits 0..15 = right neighbour (zero at the row ends and past W)
        auto ld_x = [&](const Step& t, bool live, int ci, int z, int gi, uint32_t* m)
            __attribute__((always_inline)) {
            // the step is wave-uniform; saying so keeps the resource in SGPRs
            const int n = __builtin_amdgcn_readfirstlane(t.n);
            const __amdgpu_buffer_rsrc_t xr =
                buf_rsrc_u(a.x + (int64_t)n * a.Ci * V, (uint32_t)(a.Ci * V * 2));
            const int u = 8 * gi, rr = qdiv(u, a.mWp), col = u - rr * a.Wp;
            const int h = t.h0 - 1 + rr;
            const bool ok = live && (unsigned)z < (unsigned)a.D && (unsigned)h < (unsigned)a.H;
            const uint32_t o = ok ? (uint32_t)((ci0 + ci) * (uint32_t)V + z * HW + h * a.W + col) * 2u
                                  : 0x80000000u;
            if constexpr (ELEM) {
                uint32_t e[8];
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    e[j] = buf_ld2(xr, ok && col + j < a.W ? o + 2u * j : 0x80000000u, 0);
                m[1] = e[0] | (e[1] << 16); m[2] = e[2] | (e[3] << 16);
                m[3] = e[4] | (e[5] << 16); m[4] = e[6] | (e[7] << 16);
            } else if constexpr (PART) {
                const bool full = col + 8 <= a.W;
                const uint4 v = buf_ld16(xr, full ? o : 0x80000000u, 0);
                const uint2 w = buf_ld8(xr, full ? 0x80000000u : o, 0);
                m[1] = v.x | w.x; m[2] = v.y | w.y; m[3] = v.z; m[4] = v.w;
            } else {
                const uint4 v = buf_ld16(xr, o, 0);
                m[1] = v.x; m[2] = v.y; m[3] = v.z; m[4] = v.w;
            }
            m[0] = buf_ld2(xr, ok && col > 0 ? o - 2u : 0x80000000u, 0) << 16;
            m[5] = buf_ld2(xr, ok && col + 8 < a.W ? o + 16u : 0x80000000u, 0);
        };
        auto st_x = [&](int ci, int z, int gi, const uint32_t* m) __attribute__((always_inline)) {
            unsigned char* base = xs + ci * a.cis + slot_of(z) * a.sls + gi * 16;
            uint32_t s0[4], s2[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                s0[i] = __builtin_amdgcn_alignbit(m[i + 1], m[i], 16);
                s2[i] = __builtin_amdgcn_alignbit(m[i + 2], m[i + 1], 16);
            }
            *reinterpret_cast<uint4*>(base) = make_uint4(s0[0], s0[1], s0[2], s0[3]);
            *reinterpret_cast<uint4*>(base + KWS) = make_uint4(m[1], m[2], m[3], m[4]);
            *reinterpret_cast<uint4*>(base + 2 * KWS) = make_uint4(s2[0], s2[1], s2[2], s2[3]);
        };
        auto ld_dy = [&](const Step& t, bool live, int co, int gi) __attribute__((always_inline)) {
            const int n = __builtin_amdgcn_readfirstlane(t.n);
            const __amdgpu_buffer_rsrc_t yr =
                buf_rsrc_u(a.dy + (int64_t)n * a.Co * V, (uint32_t)(a.Co * V * 2));
            const int u = 8 * gi, rr = qdiv(u, a.mWp), col = u - rr * a.Wp;
            const int h = t.h0 + rr;
            const uint32_t o =
                live && h < a.H
                    ? (uint32_t)((co0 + co) * (uint32_t)V + t.d * HW + h * a.W + col) * 2u
                    : 0x80000000u;
            if constexpr (ELEM) {
                uint32_t e[8];
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    e[j] = buf_ld2(yr, o != 0x80000000u && col + j < a.W ? o + 2u * j : 0x80000000u, 0);
                return make_uint4(e[0] | (e[1] << 16), e[2] | (e[3] << 16), e[4] | (e[5] << 16),
                                  e[6] | (e[7] << 16));
            }
            if constexpr (PART) {
                const bool full = col + 8 <= a.W;
                uint4 v = buf_ld16(yr, full ? o : 0x80000000u, 0);
                const uint2 w = buf_ld8(yr, full ? 0x80000000u : o, 0);
                v.x |= w.x;
                v.y |= w.y;
                return v;
            }
            return buf_ld16(yr, o, 0);
        };
        constexpr int NXN = (16 * (kBandSlotVox / 8) + 255) / 256;  // x groups per thread, one plane
        constexpr int NDY = 64 * (kBandK / 8) / 256;                // dy groups per thread
        struct Regs {
            uint32_t m[NXN][6];
            uint4 dy[NDY];
        };
        // A thread's staging items are the same at every step, so their
        // element offsets within a sample (x: at plane 0 of a band starting
        // at row 0; dy: likewise), their LDS offsets and their row / edge
        // flags are computed once; a step adds its wave-uniform plane and band
        // offsets.  Flags: bits 0..15 the item's row in the band, 16 live,
        // 17 a left neighbour exists, 18 a right neighbour exists, 19 eight
        // whole voxels (else four).
        uint32_t xo[NXN], xl[NXN], xf[NXN], yo[NDY], yl[NDY], yf[NDY];
        {
            const int pt = tid - 256;
#pragma unroll
            for (int q = 0; q < NXN; ++q) {
                const int it = pt + 256 * q;
                const bool live = it < 16 * XG;
                const int ci = live ? qdiv(it, a.mXG) : 0, gi = live ? it - ci * XG : 0;
                const int u = 8 * gi, rr = qdiv(u, a.mWp), col = u - rr * a.Wp;
                xo[q] = (uint32_t)(ci0 + ci) * (uint32_t)V + (uint32_t)(rr * a.W + col);
                xl[q] = (uint32_t)(ci * a.cis + gi * 16);
                const int nv = a.W - col < 8 ? (a.W - col > 0 ? a.W - col : 0) : 8;
                xf[q] = (uint32_t)rr | (live ? 1u << 16 : 0u) | (col > 0 ? 1u << 17 : 0u) |
                        (col + 8 < a.W ? 1u << 18 : 0u) | (col + 8 <= a.W ? 1u << 19 : 0u) |
                        ((uint32_t)nv << 20);
            }
#pragma unroll
            for (int q = 0; q < NDY; ++q) {
                const int it = pt + 256 * q;
                const bool live = it < 64 * YG;
                const int co = live ? qdiv(it, a.mYG) : 0, gi = live ? it - co * YG : 0;
                const int u = 8 * gi, rr = qdiv(u, a.mWp), col = u - rr * a.Wp;
                yo[q] = (uint32_t)(co0 + co) * (uint32_t)V + (uint32_t)(rr * a.W + col);
                yl[q] = (uint32_t)(co * kBandDys + gi * 16);
                const int nv = a.W - col < 8 ? (a.W - col > 0 ? a.W - col : 0) : 8;
                yf[q] = (uint32_t)rr | (live ? 1u << 16 : 0u) | (col + 8 <= a.W ? 1u << 19 : 0u) |
                        ((uint32_t)nv << 20);
            }
        }
        // one new plane (d + 1 of step t) and the dy of step t, into registers
        auto load = [&](const Step& t, Regs& R) __attribute__((always_inline)) {
            const int n = __builtin_amdgcn_readfirstlane(t.n);
            const __amdgpu_buffer_rsrc_t xr =
                buf_rsrc_u(a.x + (int64_t)n * a.Ci * V, (uint32_t)(a.Ci * V * 2));
            const __amdgpu_buffer_rsrc_t yr =
                buf_rsrc_u(a.dy + (int64_t)n * a.Co * V, (uint32_t)(a.Co * V * 2));
            const int z = t.d + 1;
            const bool zok = (unsigned)z < (unsigned)a.D;
            // uniform parts (the band's first x row is h0 - 1; unsigned wrap-around
            // cancels against the item's row term)
            const uint32_t xb = (uint32_t)(z * HW) + (uint32_t)((t.h0 - 1) * a.W);
            const uint32_t yb = (uint32_t)(t.d * HW) + (uint32_t)(t.h0 * a.W);
            const int hy = a.H - t.h0;  // dy rows left in the map
#pragma unroll
            for (int q = 0; q < NXN; ++q) {
                const uint32_t f = xf[q];
                const int rr = (int)(f & 0xffffu);
                const bool ok = (f & (1u << 16)) && zok && (unsigned)(rr - 1 + t.h0) < (unsigned)a.H;
                const uint32_t o = ok ? (xo[q] + xb) * 2u : 0x80000000u;
                uint32_t* m = R.m[q];
                if constexpr (ELEM) {
                    const int nv = (int)((f >> 20) & 15u);
                    uint32_t e[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        e[j] = buf_ld2(xr, ok && j < nv ? o + 2u * j : 0x80000000u, 0);
                    m[1] = e[0] | (e[1] << 16); m[2] = e[2] | (e[3] << 16);
                    m[3] = e[4] | (e[5] << 16); m[4] = e[6] | (e[7] << 16);
                } else if constexpr (PART) {
                    const bool full = f & (1u << 19);
                    const uint4 v = buf_ld16(xr, full ? o : 0x80000000u, 0);
                    const uint2 w = buf_ld8(xr, full ? 0x80000000u : o, 0);
                    m[1] = v.x | w.x; m[2] = v.y | w.y; m[3] = v.z; m[4] = v.w;
                } else {
                    const uint4 v = buf_ld16(xr, o, 0);
                    m[1] = v.x; m[2] = v.y; m[3] = v.z; m[4] = v.w;
                }
                m[0] = buf_ld2(xr, ok && (f & (1u << 17)) ? o - 2u : 0x80000000u, 0) << 16;
                m[5] = buf_ld2(xr, ok && (f & (1u << 18)) ? o + 16u : 0x80000000u, 0);
            }
#pragma unroll
            for (int q = 0; q < NDY; ++q) {
                const uint32_t f = yf[q];
                const int rr = (int)(f & 0xffffu);
                const bool ok = (f & (1u << 16)) && rr < hy;
                const uint32_t o = ok ? (yo[q] + yb) * 2u : 0x80000000u;
                if constexpr (ELEM) {
                    const int nv = (int)((f >> 20) & 15u);
                    uint32_t e[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        e[j] = buf_ld2(yr, ok && j < nv ? o + 2u * j : 0x80000000u, 0);
                    R.dy[q] = make_uint4(e[0] | (e[1] << 16), e[2] | (e[3] << 16),
                                         e[4] | (e[5] << 16), e[6] | (e[7] << 16));
                } else if constexpr (PART) {
                    const bool full = f & (1u << 19);
                    uint4 v = buf_ld16(yr, full ? o : 0x80000000u, 0);
                    const uint2 w = buf_ld8(yr, full ? 0x80000000u : o, 0);
                    v.x |= w.x;
                    v.y |= w.y;
                    R.dy[q] = v;
                } else {
                    R.dy[q] = buf_ld16(yr, o, 0);
                }
            }
        };
        auto commit = [&](const Step& t, const Regs& R, unsigned char* db) __attribute__((always_inline)) {
            unsigned char* xb = xs + slot_of(t.d + 1) * a.sls;
#pragma unroll
            for (int q = 0; q < NXN; ++q) {
                if (!(xf[q] & (1u << 16))) continue;
                const uint32_t* m = R.m[q];
                unsigned char* base = xb + xl[q];
                uint32_t s0[4], s2[4];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    s0[i] = __builtin_amdgcn_alignbit(m[i + 1], m[i], 16);
                    s2[i] = __builtin_amdgcn_alignbit(m[i + 2], m[i + 1], 16);
                }
                *reinterpret_cast<uint4*>(base) = make_uint4(s0[0], s0[1], s0[2], s0[3]);
                *reinterpret_cast<uint4*>(base + KWS) = make_uint4(m[1], m[2], m[3], m[4]);
                *reinterpret_cast<uint4*>(base + 2 * KWS) = make_uint4(s2[0], s2[1], s2[2], s2[3]);
            }
#pragma unroll
            for (int q = 0; q < NDY; ++q)
                if (yf[q] & (1u << 16)) *reinterpret_cast<uint4*>(db + yl[q]) = R.dy[q];
        };
        // first step of a range or band: planes d - 1 .. d + 1 and dy, synchronously
        auto stage_full = [&](const Step& t, unsigned char* db) __attribute__((always_inline)) {
            const int nx = 16 * 3 * XG;
#pragma unroll 1
            for (int it0 = ptid_now(); it0 < nx; it0 += 4 * 256) {
                uint32_t m[4][6];
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int it = it0 + 256 * i, ci = qdiv(it, a.m3XG);
                    const int rem = it - ci * 3 * XG, pl = qdiv(rem, a.mXG);
                    ld_x(t, it < nx, ci, t.d - 1 + pl, rem - pl * XG, m[i]);
                }
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const int it = it0 + 256 * i, ci = qdiv(it, a.m3XG);
                    const int rem = it - ci * 3 * XG, pl = qdiv(rem, a.mXG);
                    if (it < nx) st_x(ci, t.d - 1 + pl, rem - pl * XG, m[i]);
                }
            }
            const int pt = ptid_now();
            uint4 yv[NDY];
#pragma unroll
            for (int q = 0; q < NDY; ++q) {
                const int it = pt + 256 * q, co = qdiv(it, a.mYG);
                yv[q] = ld_dy(t, it < 64 * YG, co, it - co * YG);
            }
#pragma unroll
            for (int q = 0; q < NDY; ++q) {
                const int it = pt + 256 * q, co = qdiv(it, a.mYG);
                if (it < 64 * YG)
                    *reinterpret_cast<uint4*>(db + co * kBandDys + (it - co * YG) * 16) = yv[q];
            }
        };

        // Barrier schedule (both roles): one prologue barrier, then per step
        // one barrier, plus one more before a step that restages three planes.
        // Three register sets: the loads of step k + 3 are issued during step
        // k and written to LDS during step k + 2.
        Regs R0, R1, R2;
        if (S > 0) {
            stage_full(step_at(0), dys);
            if (S > 1 && !step_at(1).full) load(step_at(1), R1);
            if (S > 2 && !step_at(2).full) load(step_at(2), R2);
        }
        lds_barrier();
        // Rc holds step k + 1 unless that step restages; Rl takes step k + 3
        auto body = [&](int k, Regs& Rc, Regs& Rl) __attribute__((always_inline)) {
            if (k + 1 < S) {
                const Step tn = step_at(k + 1);
                unsigned char* db = dys + ((k + 1) & 1) * DYB;
                if (!tn.full) commit(tn, Rc, db);
                if (k + 3 < S) {
                    const Step tf = step_at(k + 3);
                    if (!tf.full) load(tf, Rl);
                }
                lds_barrier();
                if (tn.full) {
                    stage_full(tn, db);
                    lds_barrier();
                }
            } else {
                lds_barrier();
            }
        };
        for (int k = 0; k < S; k += 3) {
            body(k, R1, R0);
            if (k + 1 < S) body(k + 1, R2, R1);
            if (k + 2 < S) body(k + 2, R0, R2);
        }
        return;
    }

    // ---- consumer: wave w owns taps w, w + 4, ...; lane (li, kg) holds
    // voxels 32 s + 8 kg .. + 7 of output channel / input channel li
    const int li = lane & 15, kg = lane >> 4;
    f32x4 acc[NTAP][4];
#pragma unroll
    for (int j = 0; j < NTAP; ++j)
#pragma unroll
        for (int c = 0; c < 4; ++c) acc[j][c] = f32x4{0.f, 0.f, 0.f, 0.f};

    lds_barrier();
    for (int k = 0; k < S; ++k) {
        const Step t = step_at(k);
        const unsigned char* abase = dys + (k & 1) * DYB + li * kBandDys + kg * 16;
        int boff[NTAP];
#pragma unroll
        for (int jj = 0; jj < NTAP; ++jj) {
            int tp = wave + 4 * jj;
            tp = tp < KT ? tp : KT - 1;  // wave 3's seventh slot repeats tap 26, never read
            const int kd = tp / 9, kh = (tp / 3) % 3, kw = tp % 3;
            boff[jj] = kw * KWS + li * a.cis + slot_of(t.d - 1 + kd) * a.sls +
                       (kg * 8 + kh * a.Wp) * 2;
        }
        constexpr int G = NK * NTAP;
        constexpr int LA = 3;
        F16B A[2][4], B[4];
#pragma unroll
        for (int ct = 0; ct < 4; ++ct)
            A[0][ct].u = *reinterpret_cast<const uint4*>(abase + ct * 16 * kBandDys);
#pragma unroll
        for (int g = 0; g < LA; ++g)
            B[g].u = *reinterpret_cast<const uint4*>(xs + boff[g % NTAP] + (g / NTAP) * 64);
#pragma unroll
        for (int g = 0; g < G; ++g) {
            const int s_ = g / NTAP, jj = g % NTAP;
            if (g + LA < G) {
                const int gn = g + LA;
                B[gn % 4].u =
                    *reinterpret_cast<const uint4*>(xs + boff[gn % NTAP] + (gn / NTAP) * 64);
            }
            if (jj == 3 && s_ + 1 < NK) {
#pragma unroll
                for (int ct = 0; ct < 4; ++ct)
                    A[(s_ + 1) & 1][ct].u = *reinterpret_cast<const uint4*>(
                        abase + ct * 16 * kBandDys + (s_ + 1) * 64);
            }
#pragma unroll
            for (int ct = 0; ct < 4; ++ct)
                acc[jj][ct] = mfma(A[s_ & 1][ct], B[g % 4], acc[jj][ct]);
            __builtin_amdgcn_sched_barrier(0);
        }
        lds_barrier();
        if (k + 1 < S && step_at(k + 1).full) lds_barrier();
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

// dst[i] = round((sum over splits, in split order, of part[split][i]) + bias[co]
// (+ dst[i] when accumulating)): one rounding, as the unsplit epilogue.
__global__ __launch_bounds__(256) void brick_split_reduce(const float* __restrict__ part,
                                                          int nsplit, int64_t count, int Ct,
                                                          int64_t V, const float* __restrict__ bias,
                                                          bf16* __restrict__ dst, int accumulate) {
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= count) return;
    float s = part[i];
    for (int z = 1; z < nsplit; ++z) s += part[(int64_t)z * count + i];
    if (bias) s += bias[(int)((i / V) % Ct)];
    if (accumulate) s += bf2f(dst[i]);
    dst[i] = f2bf(s);
}

// ---------------------------------------------------------------- dispatch
bool brick_fd_ok(const ConvGeom& g, rat3d_dtype dt, bool dgrad) {
    if (dt != RAT3D_BF16 || g.s != 1) return false;
    if (!((g.k == 3 && g.p == 1) || (g.k == 1 && g.p == 0))) return false;
    const int cs = dgrad ? g.Co : g.Ci, ct = dgrad ? g.Ci : g.Co;
    // one sample's source and target channels are addressed with 32-bit
    // byte offsets
    const int64_t vox_bytes = (int64_t)g.D * g.H * g.W * 2;
    return cs % 32 == 0 && ct % 32 == 0 && cs * vox_bytes < ((int64_t)1 << 31) &&
           ct * vox_bytes < ((int64_t)1 << 31);
}

// Row bands take maps up to 56 columns wide (W a multiple of 4): hb rows of
// pitch Wp with hb * Wp <= NK * 32 and (hb + 2) * Wp <= 288 (the LDS slot
// bound); NK in {6, 4} is picked for the fewest K steps per plane.
struct BandCfg {
    int hb = 0, nk = 0, Wp = 0;
};
static BandCfg band_cfg(const ConvGeom& g) {
    BandCfg c;
    const int Wp = (g.W + 7) & ~7;
    // staging addresses one sample's tensor with 32-bit byte offsets
    const int64_t v2 = (int64_t)g.D * g.H * g.W * 2;
    if (Wp > 56 || (int64_t)g.Ci * v2 >= ((int64_t)1 << 31) ||
        (int64_t)g.Co * v2 >= ((int64_t)1 << 31))
        return c;
    // element-loaded widths (W % 4 != 0) only on maps of 128 voxels or more:
    // below that the kernel's fixed costs (prologue, one partial block per
    // workgroup) exceed the gather kernel's time (3x4x3: 47 vs 39 us at 256
    // channels, measured; 6x7x6: 69 vs 128 us)
    if (g.W % 4 != 0 && (int64_t)g.D * g.H * g.W < 128) return c;
    int64_t best = -1;
    // least work per plane: each band costs its nk K steps plus a fixed
    // overhead of about two (barrier, staging of hb + 2 rows); two or one K
    // step of 32 voxels serve the smallest planes (a 6 x 7 plane at pitch 8
    // fills 56 of 64 slots)
    for (int nk : {6, 4, 2, 1}) {
        const int a = nk * 32 / Wp, b = kBandSlotVox / Wp - 2;
        const int hb = a < b ? a : b;
        if (hb < 1) continue;
        const int64_t cost = ceil_div(g.H, hb) * (nk + 2);
        if (best < 0 || cost < best) {
            best = cost;
            c.hb = hb;
            c.nk = nk;
            c.Wp = Wp;
        }
    }
    return c;
}

bool brick_wgrad_ok(const ConvGeom& g, rat3d_dtype dt) {
    return dt == RAT3D_BF16 && g.s == 1 && g.k == 3 && g.p == 1 && g.Ci % 16 == 0 &&
           g.Co % 64 == 0 && (g.W % 8 == 0 || band_cfg(g).hb > 0);
}

// Tile plan of a brick pass: 64-channel tiles unless that leaves most CUs
// idle (small volumes: then 32-channel tiles double the workgroups), and a
// split over the 32-channel source chunks when the tiles are fewer than the
// CUs and splitting at least halves the busiest CU's step count (a smaller
// gain does not pay for writing and summing the fp32 partials).
struct BrickPlan {
    int nt, cogs, ntiles, nsplit;  // ntiles: spatial tiles x channel groups
};
static BrickPlan brick_plan(const ConvGeom& g, bool dgrad) {
    const int cs = dgrad ? g.Co : g.Ci, ct = dgrad ? g.Ci : g.Co;
    const int64_t sp_tiles =
        (int64_t)g.N * ceil_div(g.D, kBD) * ceil_div(g.H, kBH) * ceil_div(g.W, kBW);
    const int cus = device_cus();
    BrickPlan p;
    p.nt = (ct % 64 == 0 && sp_tiles * (ct / 64) >= cus / 2) ? 4 : 2;
    p.cogs = ct / (p.nt * 16);
    p.ntiles = (int)(sp_tiles * p.cogs);
    p.nsplit = 1;
    if (g.k == 3 && p.ntiles < cus) {
        const int nchunk = cs / 32;
        auto steps = [&](int ns) { return ceil_div((int64_t)p.ntiles * ns, cus) * (nchunk / ns); };
        int64_t best = steps(1);
        for (int ns = 2; ns <= nchunk && nchunk % ns == 0; ns *= 2) {
            const int64_t st = steps(ns);
            if (st * 2 <= steps(1) && st < best) {
                best = st;
                p.nsplit = ns;
            }
        }
    }
    return p;
}

static size_t brick_prepared_bytes(const ConvGeom& g) {
    return ((size_t)g.Co * g.Ci * g.k * g.k * g.k * 2 + 255) & ~(size_t)255;
}

size_t brick_fd_ws(const ConvGeom& g, bool dgrad) {
    const BrickPlan p = brick_plan(g, dgrad);
    const size_t part = p.nsplit > 1 ? (size_t)p.nsplit * g.N * (dgrad ? g.Ci : g.Co) *
                                           ((size_t)g.D * g.H * g.W) * sizeof(float)
                                     : 0;
    return brick_prepared_bytes(g) + part;
}

static int64_t wgrad_steps(const ConvGeom& g) {
    const int hb = band_cfg(g).hb;
    if (hb > 0) return (int64_t)g.N * ceil_div(g.H, hb) * g.D;
    return (int64_t)g.N * ceil_div(g.H, kWH) * ceil_div(g.W, kWW) * ceil_div(g.D, 2);
}

static int wgrad_ranges(const ConvGeom& g) {
    // one workgroup per CU: the (C_in, C_out) groups times the step ranges
    const int64_t groups = (int64_t)(g.Ci / 16) * (g.Co / 64);
    int64_t r = device_cus() / groups;
    const int64_t ns = wgrad_steps(g);
    if (r > ns) r = ns;
    if (r < 1) r = 1;
    return (int)r;
}

size_t brick_wgrad_ws(const ConvGeom& g) {
    const int R = wgrad_ranges(g);
    return (size_t)R * (g.Ci / 16) * (g.Co / 64) * kWgPart * sizeof(float);
}

rat3d_status brick_prep_weights(const ConvGeom& g, bool dgrad, const void* w, void* wt,
                                hipStream_t st) {
    const PrepJob job{g, dgrad, w, wt};
    return brick_prep_weights_batch(&job, 1, st);
}

rat3d_status conv_fd_brick(const ConvGeom& g, bool dgrad, const void* src, const void* w,
                           const float* bias, void* dst, int accumulate, void* ws,
                           hipStream_t st, bool w_prepared) {
    const bf16* wt = (const bf16*)w;
    if (!w_prepared) {
        const rat3d_status s = brick_prep_weights(g, dgrad, w, ws, st);
        if (s != RAT3D_OK) return s;
        wt = (const bf16*)ws;
    }
    if (pw_fd_ok(g, RAT3D_BF16, dgrad))
        return conv_fd_pw(g, dgrad, src, wt, bias, dst, accumulate, st);
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
    const BrickPlan plan = brick_plan(g, dgrad);
    const int nt = plan.nt;
    a.cogs = plan.cogs;
    a.nsplit = plan.nsplit;
    a.cps = (a.Cs / 32) / plan.nsplit;
    a.ntiles = plan.ntiles * plan.nsplit;
    a.part = (float*)((char*)ws + brick_prepared_bytes(g));
    // one persistent workgroup per CU (fewer when there are fewer items)
    const int grid = a.ntiles < device_cus() ? a.ntiles : device_cus();
    // one tag (and one kernel symbol) per variant, so that live timings and
    // profiler counters describe the same launches
    const bool acc = accumulate != 0;
    const char* tag = g.k == 3 ? (dgrad ? (acc ? "conv_brick3_dgrad_acc" : "conv_brick3_dgrad")
                                        : "conv_brick3_fwd")
                               : (dgrad ? (acc ? "conv_brick1_dgrad_acc" : "conv_brick1_dgrad")
                                        : "conv_brick1_fwd");
    char tagbuf[48];
    if (nt == 2 || plan.nsplit > 1) {
        snprintf(tagbuf, sizeof tagbuf, "%s%s%s", tag, nt == 2 ? "_c32" : "",
                 plan.nsplit > 1 ? "_split" : "");
        tag = tagbuf;
    }
    ProfScope ps(tag, st, conv_flops(g), conv_bytes(g, 2));
#define RAT3D_FD(K, N, R)                                                          \
    do {                                                                           \
        if (dgrad) {                                                               \
            if (acc) conv_brick_fd<K, N, R, true, true><<<grid, 512, 0, st>>>(a);  \
            else conv_brick_fd<K, N, R, false, true><<<grid, 512, 0, st>>>(a);     \
        } else {                                                                   \
            if (acc) conv_brick_fd<K, N, R, true, false><<<grid, 512, 0, st>>>(a); \
            else conv_brick_fd<K, N, R, false, false><<<grid, 512, 0, st>>>(a);    \
        }                                                                          \
    } while (0)
    if (g.k == 3) {
        if (nt == 4) RAT3D_FD(3, 4, 2);
        else RAT3D_FD(3, 2, 1);
    } else {
        if (nt == 4) RAT3D_FD(1, 4, 2);
        else RAT3D_FD(1, 2, 1);
    }
#undef RAT3D_FD
    RAT3D_LAUNCH_CHECK();
    if (plan.nsplit > 1) {
        const int64_t V = (int64_t)g.D * g.H * g.W, count = (int64_t)g.N * a.Ct * V;
        brick_split_reduce<<<(unsigned)ceil_div(count, 256), 256, 0, st>>>(
            a.part, plan.nsplit, count, a.Ct, V, dgrad ? nullptr : bias, (bf16*)dst, accumulate);
        RAT3D_LAUNCH_CHECK();
    }
    return RAT3D_OK;
}

rat3d_status conv_wgrad_brick(const ConvGeom& g, const void* x, const void* dy, float* dw,
                              int accumulate, void* ws, hipStream_t st) {
    const int64_t nsteps = wgrad_steps(g);
    const int R = wgrad_ranges(g);
    const int spr = (int)ceil_div(nsteps, R);
    const int Rreal = (int)ceil_div(nsteps, spr);
    const int cigs = g.Ci / 16, cogs = g.Co / 64;
    const BandCfg bc = band_cfg(g);
    const int hb = bc.hb;
    if (hb > 0) {
        WbArgs a;
        a.x = (const bf16*)x;
        a.dy = (const bf16*)dy;
        a.part = (float*)ws;
        a.N = g.N;
        a.Ci = g.Ci;
        a.Co = g.Co;
        a.D = g.D;
        a.H = g.H;
        a.W = g.W;
        a.Wp = bc.Wp;
        a.hb = hb;
        a.nb = (int)ceil_div(g.H, hb);
        a.nsteps = (int)nsteps;
        a.spr = spr;
        a.cigs = cigs;
        a.cogs = cogs;
        a.sls = (hb + 2) * bc.Wp * 2;
        // input-channel stride an odd multiple of 32 bytes: the 16 channels of
        // one operand read (one per lane of a 16-lane group) then take one LDS
        // pass (a stride of 16 mod 128 measured two)
        a.cis = ((4 * a.sls + 127) & ~127) + 32;
        if (a.cis > kBandCisMax) {  // band_cfg keeps (hb + 2) * Wp <= kBandSlotVox
            set_error("conv3d wgrad: band slot of %d bytes exceeds the LDS layout", a.cis);
            return RAT3D_EINVAL;
        }
        const int XG = (hb + 2) * bc.Wp / 8, YG = hb * bc.Wp / 8;
        auto magic = [](int d) { return (uint32_t)(((1u << 20) + d - 1) / d); };
        a.mWp = magic(bc.Wp);
        a.mXG = magic(XG);
        a.m3XG = magic(3 * XG);
        a.mYG = magic(YG);
        // staging mode: whole 8-voxel groups, a half-filled last group, or
        // element loads (widths that are not a multiple of 4)
        const int mode = (g.W & 7) == 0 ? 0 : ((g.W & 3) == 0 ? 1 : 2);
        char tag[48];
        snprintf(tag, sizeof tag, "conv_band3_wgrad%s%s",
                 bc.nk == 6 ? "" : bc.nk == 4 ? "_k128" : bc.nk == 2 ? "_k64" : "_k32",
                 mode == 1 ? "_w4" : mode == 2 ? "_elem" : "");
        ProfScope ps(tag, st, conv_flops(g), conv_bytes(g, 2));
        const unsigned grid = (unsigned)((int64_t)Rreal * cigs * cogs);
#define RAT3D_BAND(NK)                                                           \
    do {                                                                         \
        if (mode == 0) conv_band_wgrad<NK, 0><<<grid, 512, 0, st>>>(a);          \
        else if (mode == 1) conv_band_wgrad<NK, 1><<<grid, 512, 0, st>>>(a);     \
        else conv_band_wgrad<NK, 2><<<grid, 512, 0, st>>>(a);                    \
    } while (0)
        if (bc.nk == 6) RAT3D_BAND(6);
        else if (bc.nk == 4) RAT3D_BAND(4);
        else if (bc.nk == 2) RAT3D_BAND(2);
        else RAT3D_BAND(1);
#undef RAT3D_BAND
        RAT3D_LAUNCH_CHECK();
    } else {
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
        a.tds = (int)ceil_div(g.D, 2);
        a.th = (int)ceil_div(g.H, kWH);
        a.tw = (int)ceil_div(g.W, kWW);
        a.nsteps = (int)nsteps;
        a.spr = spr;
        a.cigs = cigs;
        a.cogs = cogs;
        ProfScope ps("conv_brick3_wgrad", st, conv_flops(g), conv_bytes(g, 2));
        conv_brick_wgrad<3><<<(unsigned)((int64_t)Rreal * cigs * cogs), 512, 0, st>>>(a);
        RAT3D_LAUNCH_CHECK();
    }
    const int groups = cigs * cogs;
    const int64_t count = (int64_t)groups * kWgPart;
    ProfScope ps("wgrad_reduce", st, 0.0,
                 4.0 * (count * Rreal + (double)g.Co * g.Ci * 27 * (1 + accumulate)));
    wgrad_brick_reduce<<<(unsigned)ceil_div(count, 256), 256, 0, st>>>(
        (const float*)ws, Rreal, groups, cigs, g.Ci, dw, accumulate);
    RAT3D_LAUNCH_CHECK();
    return RAT3D_OK;
}

}  // namespace rat3d
