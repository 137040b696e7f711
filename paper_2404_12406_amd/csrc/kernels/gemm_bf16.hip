// bf16 implicit-GEMM kernels for gfx950: the fast path of the three
// contractions of a layer that is linear in input and weight (Sec. 2.2.1 of
// the paper) -- forward, input gradient (needs W only) and weight gradient
// (needs x only) -- for NHWC activations and KRSC filters.  The GEMM views
// and the stride-phase split of the input gradient are those of igemm.hip.
//
// Data movement (per block of NW = 4 or 8 waves in a WR x WC grid):
//  * operands go from HBM straight into LDS with buffer_load_dwordx4 ... lds
//    (no VGPR staging).  Each lane computes the byte offset of its 16-byte
//    chunk; lanes that fall into padding, a ragged tail or a missing tap use
//    an offset beyond the buffer's range and the hardware writes zeros.
//  * the reduction step is BK = 64: a K-contiguous tile row is 128 bytes, one
//    full cache line, so every load instruction moves eight whole lines
//    (BK = 32 rows are half lines and cost the vector-memory path twice the
//    work per byte).
//  * STAGES LDS buffers form a ring with one barrier per BK step; within a
//    step the fragments of the next 16-k slice are read from LDS while the
//    MFMAs of the current slice run (register double buffering per slice).
//  * operands contiguous along k are stored [row][k] with 16-byte chunks
//    XOR-swizzled by row and read as MFMA fragments with ds_read_b128;
//    operands contiguous along m/n are stored [k][mn] with 16-byte slots
//    swizzled by k-row and read with ds_read_b64_tr_b16, which transposes a
//    16 x 4 block of b16 within each 16-lane group (two reads = 8 k values).
//  * v_mfma_f32_32x32x16_bf16 with the B fragment as first operand, so each
//    lane ends with groups of 4 consecutive output columns of one row; the
//    epilogue packs them to bf16, stages the tile through LDS and writes
//    16-byte vectors (fp32 split-K partials are stored as float4 directly).
//  * weight gradient: long reductions are split over grid z; when the bias
//    gradient is requested too, the waves that load dy (operand A) add up
//    its rows from their fragments -- the bias gradient costs no extra read.
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include <hip/hip_ext.h>

#include "common.h"
#include "limits.h"
#include "../device.h"

namespace ms {
namespace g2 {

typedef __attribute__((address_space(3))) void lds_void_t;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16_t;

// kDgrad reads the filter from a transposed copy Wt[C][R][S][K] (both
// operands K-contiguous); kDgradN reads W[K][R][S][C] in place as an
// M/N-contiguous operand (no copy, transposing LDS reads).
enum Mode { kFwd = 0, kDgrad = 1, kWgrad = 2, kDgradN = 3 };

constexpr int BK = 64;                   // reduction step (elements)

struct Args {
    const bf16 *a;
    const bf16 *b;
    bf16 *c;              // output (or nullptr when the output is fp32 partials)
    float *part;          // split-K partials: part_stride floats per split (nullptr: splits == 1)
    float *dbpart;        // WGRAD fused bias-gradient partials [splits][M] (nullptr: off)
    float *cspart;        // unit-geometry DGRAD: column sums of dy (the bias gradient),
                          // one partial row per (row tile, summing wave) (nullptr: off)
    int cs_cw;            // columns of dy per block column (a multiple of 8)
    int64_t part_stride;  // FWD/WGRAD: M*N; DGRAD: N*H*W*C (partials indexed by dx pixel)
    const bf16 *bias;     // FWD / DGRAD per-column bias (nullptr: none; DGRAD: the
                          // transposed convolution's forward)
    ConvGeom g;
    int M, N, K;          // GEMM extents (DGRAD: bounds over phases)
    int ntm, ntn;
    int ldc;              // bf16 output row stride in elements (0: N); a launch that covers
                          // a column range of a wider output passes the full width
    int k_split, splits;  // reduction range per split (a multiple of BK) and split count
    uint32_t a_bytes, b_bytes;
};

struct Phase {
    int fh, fw, h0, w0, Hp, Wp, Rp, Sp, dh, dw;
};

__device__ __forceinline__ Phase make_phase(const ConvGeom &g, int z) {
    Phase f;
    f.fh = z / g.sw;
    f.fw = z % g.sw;
    f.h0 = ((f.fh - g.ph) % g.sh + g.sh) % g.sh;
    f.w0 = ((f.fw - g.pw) % g.sw + g.sw) % g.sw;
    f.Hp = f.h0 < g.H ? (g.H - f.h0 + g.sh - 1) / g.sh : 0;
    f.Wp = f.w0 < g.W ? (g.W - f.w0 + g.sw - 1) / g.sw : 0;
    f.Rp = f.fh < g.R ? (g.R - f.fh + g.sh - 1) / g.sh : 0;
    f.Sp = f.fw < g.S ? (g.S - f.fw + g.sw - 1) / g.sw : 0;
    f.dh = (f.h0 + g.ph - f.fh) / g.sh;
    f.dw = (f.w0 + g.pw - f.fw) / g.sw;
    return f;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(p), (short)0, (int)bytes, 0x00020000);
}

// One 16-byte LDS-DMA load: lane l's 16 bytes from byte offset `off` of the
// buffer land at lds + 16 l (M0 holds the wave's LDS base).
//
// Contractions with an M/N-contiguous operand (ASM = true) issue it through
// inline assembly so that the compiler does not track it: for a pending
// LDS-DMA load the compiler puts a wait for every outstanding vector-memory
// operation in front of each transposing LDS read (ds_read_b64_tr_b16),
// which drains all refill loads in flight at every slice.  The others keep
// the builtin, whose loads the scheduler can spread between the MFMAs.
// Ordering in the assembly form is the kernel's own:
//  * completion: its vmcnt waits before each barrier;
//  * a refill writes a stage no wave reads until after the next barrier, and
//    a volatile asm statement never moves across the barrier;
//  * block_sync() tells the compiler that LDS may have changed, so no LDS
//    value read before a barrier is reused after it.
// M0 is reserved by the compiler and no other instruction of these kernels
// reads it.
// (The offset is computed into a named value first: passing a conditional
// expression straight into the builtin inside a kernel template makes the
// host pass drop the kernel's launch stub.)
template <bool ASM>
__device__ __forceinline__ void dma16(__amdgpu_buffer_rsrc_t r, char *lds, uint32_t off) {
    if constexpr (ASM) {
        const uint32_t base = (uint32_t)(uintptr_t)(lds_void_t *)lds;
        asm volatile("s_mov_b32 m0, %1\n\tbuffer_load_dwordx4 %0, %2, 0 offen lds" ::"v"(off), "s"(base), "s"(r));
    } else {
        __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t *)lds, 16, off, 0, 0, 0);
    }
}

// Workgroup barrier; with untracked LDS-DMA loads it is also a compiler-level
// memory fence (the barrier builtin alone does not stop the compiler from
// keeping LDS values across it).
template <bool ASM>
__device__ __forceinline__ void block_sync() {
    if constexpr (ASM) __atomic_signal_fence(__ATOMIC_SEQ_CST);
    __builtin_amdgcn_s_barrier();
    if constexpr (ASM) __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// s_waitcnt with only vmcnt constrained (gfx9 encoding: vmcnt[3:0] | [15:14],
// expcnt[6:4] = 7, lgkmcnt[11:8] = 15).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
__device__ __forceinline__ void wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xc07f); }

// 16-byte chunk swizzle of a K-contiguous tile row (128 bytes = 8 chunks).
// 16 consecutive rows reading the same logical chunk land on 16 distinct
// 16-byte bank groups (the LDS serves 256 bytes per clock).
__device__ __forceinline__ int swz_k(int row) { return (row & 7) ^ ((row >> 3) & 1); }

// Slot swizzle of an M/N-contiguous tile k-row ([k][mn], 16-byte slots).
// A transposed read serves 32 lanes at a time: two 16-lane groups that each
// read 4 k-rows x 2 adjacent slots, the second group 2 slots to the right.
// Rows of 16 or more slots start on the same bank, so the XOR must spread
// the 4 rows by 4 slots (the 32 lanes then cover 16 distinct slots = all 64
// banks); rows of 8 slots alternate between the two bank halves and an XOR
// by 2 suffices.  Both keep the slot pair of a group adjacent.
template <int SPR>
__device__ __forceinline__ int swz_m(int krow) {
    if constexpr (SPR >= 16) return (krow & 3) << 2;
    else return (krow & 3) << 1;
}

// MFMA fragment (8 k values of one m/n index) from a [BK k][R mn] tile for
// the 32x32x16 shape: lane l needs column mn0 + l%32 at k-rows
// 16*sub + 8*(l/32) .. +7.  ds_read_b64_tr_b16 works per 16-lane group
// g = l/16: lane 16g + r addresses k-row kb + 4h + r/4 at columns
// cb + 4*(r%4) .. +3 (kb = 16*sub + 8*(g/2), cb = mn0 + 16*(g%2)) and, after
// the in-group transpose, holds column cb + r of k-rows kb + 4h .. kb+4h+3.
template <int R>
__device__ __forceinline__ bf16x8 frag_mn(const char *base, int mn0, int sub, int lane) {
    constexpr int SPR = R / 8;
    const int g = lane >> 4, r = lane & 15;
    const int kb = 16 * sub + 8 * (g >> 1), cb = mn0 + 16 * (g & 1);
    bf16x8 v;
    v4i16 *pv = reinterpret_cast<v4i16 *>(&v);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int krow = kb + 4 * h + (r >> 2);
        const int mn = cb + 4 * (r & 3);
        const int pos = (mn >> 3) ^ swz_m<SPR>(krow);
        const int off = krow * (R * 2) + (pos << 4) + ((mn & 7) << 1);
        pv[h] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_t *)(base + off));
    }
    return v;
}

// Fragment from a row-major [row][BK] tile (128-byte rows, swizzled 16-byte
// chunks): lane l reads row `row` (= tile row + l%32), chunk 2*sub + l/32.
__device__ __forceinline__ bf16x8 frag_kc(const char *base, int row, int sub, int lane) {
    const int chunk = 2 * sub + (lane >> 5);
    const int off = row * (BK * 2) + ((chunk ^ swz_k(row)) << 4);
    return *reinterpret_cast<const bf16x8 *>(base + off);
}

// Column sums of dy for the bias gradient, taken by a unit-geometry input
// gradient (there A = dy: row m holds the K output channels of pixel m).
// Block (tm, tn) adds rows m0 .. m0+BM-1 for columns [tn*cw, tn*cw + cw) of
// K; nwc waves take part, wave w writing partial row tm*nwc + w of part
// ([rows][K] fp32).  Lane t = 64w + l of the nwc*64 owns column vector
// t % cvp (8 channels) of each pass of 8*cvp columns and walks the rows
// t / cvp + i * rgs (rgs = nwc*64 / cvp), NB loads in flight; the lanes of a
// wave that share a column vector meet by shuffles.  Loads go through the
// buffer descriptor of dy with out-of-range rows and columns sent past its
// end, so they read zeros.  The data was read by this block's main loop
// moments earlier.  issue() may be called first (the first batch of the
// first pass, e.g. before an epilogue); run() then starts from it.
template <int NB>
struct DyColumnSums {
    __amdgpu_buffer_rsrc_t ra;
    int M, K, m0, BM, kb, ncv, cvp, cvl, rg, rgs;
    bool on;
    u32x4 v[NB];

    __device__ __forceinline__ DyColumnSums(__amdgpu_buffer_rsrc_t ra_, int M_, int K_, int m0_, int BM_, int tn,
                                            int cw, int w, int nwc, int lane)
        : ra(ra_), M(M_), K(K_), m0(m0_), BM(BM_) {
        kb = tn * cw;
        on = kb < K;   // uniform over the block
        ncv = on ? (min(cw, K - kb) + 7) / 8 : 0;
        cvp = 1;
        while (cvp < ncv && cvp < 64) cvp <<= 1;
        const int t = w * 64 + lane;
        cvl = t % cvp;
        rg = t / cvp;
        rgs = nwc * 64 / cvp;
    }
    __device__ __forceinline__ void issue(int c0, int r0) {
        const int k = kb + (c0 + cvl) * 8;
        const bool kin = c0 + cvl < ncv && k < K;
#pragma unroll
        for (int i = 0; i < NB; ++i) {
            const int r = r0 + i * rgs, m = m0 + r;
            const bool ok = kin && r < BM && m < M;
            const uint32_t off = ok ? ((uint32_t)m * (uint32_t)K + (uint32_t)k) * 2u : kOOB;
            v[i] = __builtin_amdgcn_raw_buffer_load_b128(ra, (int)off, 0, 0);
        }
    }
    __device__ __forceinline__ void add(float (&acc)[8]) const {
#pragma unroll
        for (int i = 0; i < NB; ++i)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                acc[2 * q] += __uint_as_float(v[i][q] << 16);
                acc[2 * q + 1] += __uint_as_float(v[i][q] & 0xffff0000u);
            }
    }
    __device__ __forceinline__ void run(bool issued, int w, int nwc, int tm, int lane, float *__restrict__ part) {
        if (!on) return;
        for (int c0 = 0; c0 < ncv; c0 += cvp) {
            float acc[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) acc[e] = 0.f;
            for (int r0 = rg; r0 < BM; r0 += NB * rgs) {
                if (!(issued && c0 == 0 && r0 == rg)) issue(c0, r0);
                add(acc);
            }
            for (int sh = cvp; sh < 64; sh <<= 1)
#pragma unroll
                for (int e = 0; e < 8; ++e) acc[e] += __shfl_xor(acc[e], sh);
            const int k = kb + (c0 + cvl) * 8;
            if (lane < cvp && c0 + cvl < ncv && k < K) {
                float *dst = part + (size_t)(tm * nwc + w) * K + k;
                *reinterpret_cast<floatx4 *>(dst) = floatx4{acc[0], acc[1], acc[2], acc[3]};
                *reinterpret_cast<floatx4 *>(dst + 4) = floatx4{acc[4], acc[5], acc[6], acc[7]};
            }
        }
    }
};

// KG k-groups of WR x WC waves: group g computes the whole block tile from
// the 16-k slices 2g and 2g+1 of every BK step (KG = 2), and the groups add
// their accumulators through LDS at the end.  Each wave then keeps a 64 x 64
// tile (one fragment read per MFMA) with two waves per SIMD.
template <int MODE, int BM, int BN, int WR, int WC, int STAGES, int KG = 1>
struct Cfg {
    static constexpr int NW = WR * WC * KG, NT = NW * 64;
    static constexpr bool A_KC = MODE != kWgrad;
    static constexpr bool B_KC = MODE == kFwd || MODE == kDgrad;   // kDgrad: W transposed to [C][R][S][K]
    static constexpr int A_BYTES = BM * BK * 2, B_BYTES = BN * BK * 2;
    static constexpr int STAGE_BYTES = A_BYTES + B_BYTES;
    static constexpr int LDS_BYTES = STAGES * STAGE_BYTES;
    // forward: the block's bias columns, loaded once into LDS past the stages
    // (one 16-byte load per lane of wave 0)
    static constexpr int BIAS_OFF = LDS_BYTES;
    // 1 KB load instructions per tile, and per wave: where the waves do not
    // divide A's (12 waves, 32 KB), the last waves' spare slots load zeros
    // into a dummy area past everything else, so that every wave issues the
    // same number of loads per stage (the vmcnt waits count them)
    static constexpr int A_INS = A_BYTES / 1024, B_INS = B_BYTES / 1024;
    static constexpr int NIA = (A_INS + NW - 1) / NW;
    static constexpr int NIB = B_INS / NW;
    static constexpr bool A_SPARE = NIA * NW != A_INS;
    static constexpr int DUMMY_OFF = LDS_BYTES + (MODE == kFwd ? 64 * 16 : 0);
    static constexpr int SMEM_BYTES = DUMMY_OFF + (A_SPARE ? 1024 : 0);
    static constexpr int WM = BM / WR, WN = BN / WC;
    static constexpr int TM = WM / 32, TN = WN / 32;   // 32x32 MFMA tiles per wave
    static constexpr int NSUB = BK / 16;               // 16-k slices per step
    static constexpr int EPI_PITCH = WN + 8;           // bf16 elements per staged row
    static constexpr int EPI_ROWS = 32;                // rows staged per pass
    static_assert(NIA >= 1 && NIB >= 1 && A_INS * 1024 == A_BYTES && NIB * NW * 1024 == B_BYTES, "load split");
    static_assert(!A_SPARE || (A_KC && MODE != kWgrad), "spare A load slots: k-contiguous A only");
    static_assert(TM >= 1 && TN >= 1 && WM % 32 == 0 && WN % 32 == 0, "wave tile");
    static_assert(NW * EPI_ROWS * EPI_PITCH * 2 <= LDS_BYTES, "epilogue staging must fit in LDS");
    static_assert(SMEM_BYTES <= 160 * 1024, "LDS");
    static_assert(BN * 2 <= 64 * 16, "bias columns fit the bias area");
    static_assert(KG == 1 || (KG == 2 && STAGES >= 3 && MODE != kWgrad), "k-groups: spread pipeline, no weight gradient");
    // block widths that are not a power of two (192, 288) only with both operands
    // k-contiguous: the transposing reads' slot swizzle needs 2^n slots a row
    static_assert((BN & (BN - 1)) == 0 || (A_KC && B_KC), "a 192- or 288-wide tile reads k-contiguous operands only");
    static_assert(KG == 1 || (WR * WC) * (WM / 32) * (WN / 32) * 16 * 64 * 4 <= LDS_BYTES, "k-group partials fit LDS");
};

template <int MODE, int BM, int BN, int WR, int WC, int STAGES, int OCC, bool UNIT, int KG = 1, bool TS = false>
__global__ __launch_bounds__(WR * WC * KG * 64, OCC) void gemm_kernel(const Args P) {
    __shared__ __attribute__((aligned(1024))) char smem[Cfg<MODE, BM, BN, WR, WC, STAGES, KG>::SMEM_BYTES];
    const int bx = (int)blockIdx.x, bz = (int)blockIdx.z;
#include "gemm_block_body.inc"
}

// The same tile body as a device function, for the paired launch below: the
// LDS comes in from the kernel, which holds one arena for both tiles.
template <int MODE, int BM, int BN, int WR, int WC, int STAGES, bool UNIT, int KG, bool TS>
__device__ __forceinline__ void gemm_pair_block(const Args &P, char *smem, const int bx, const int bz) {
#include "gemm_block_body.inc"
}

// A column-split unit-geometry contraction in one launch: block b computes
// tile b of the leading columns (P1, on the 256 x 256 tile), then tile b of
// the remaining columns (P2, on 256 x 128), with the same number of tiles
// in both parts (one per CU).  Against two launches, a block starts its
// second tile as soon as its first is written instead of after the slowest
// block of the first launch, the kernel-end write-back and the next
// dispatch.  The XCD-aware tile order gives a block the same rows in both
// parts, so its A rows are still in its XCD's L2.  Both parts are one
// k-group tiles: every wave runs both bodies to the end, so the barrier
// between them (LDS reuse) is met by all.
template <int MODE>
__global__ __launch_bounds__(512, 1) void gemm_pair_kernel(const Args P1, const Args P2) {
    using G1 = Cfg<MODE, 256, 256, 2, 4, 2>;
    using G2 = Cfg<MODE, 256, 128, 2, 4, 3>;
    static_assert(G1::NW == 8 && G2::NW == 8, "both parts are 8-wave tiles");
    constexpr int SM = G1::SMEM_BYTES > G2::SMEM_BYTES ? G1::SMEM_BYTES : G2::SMEM_BYTES;
    __shared__ __attribute__((aligned(1024))) char smem[SM];
    gemm_pair_block<MODE, 256, 256, 2, 4, 2, true, 1, false>(P1, smem, (int)blockIdx.x, 0);
    __syncthreads();   // every wave is done with the first tile's LDS
    gemm_pair_block<MODE, 256, 128, 2, 4, 3, true, 1, false>(P2, smem, (int)blockIdx.x, 0);
}

// ---------------------------------------------------------------- halo convolution
// A stride-1 convolution of a 64-channel input whose filter fits in LDS: the
// 3x3 64 -> 64 layers of a ResNet stage 1 (forward, and input gradient as the
// correlation of dy with the flipped, transposed filter) and the stride-1
// 4x4 form of the 3-channel stem's input gradient (2x2 pixel blocks).  The
// implicit GEMM streams every input pixel through L2 once per tap (9 to 16
// times the tensor), which is what bounds those layers.  Here a persistent
// block keeps the whole filter in LDS and loads each output tile's input
// neighbourhood (the tile plus R-1 rows and S-1 columns of halo) once, with
// the next tile's halo loading into a second buffer while the current tile's
// MFMAs run; every tap's A fragments are read from that copy.
//
// in[n][h][w][64] (NHWC); filt[NO][TAPS][64]: row n of tap t holds output
// channel n's weights over the 64 input channels (flip: output tap t reads
// filter tap TAPS-1-t); out[n][p][q][NO], out[p][q] = bias + sum over taps
// (r, s) of filt . in[p - ph + r][q - pw + s], zero outside the input.
// A block is KG k-groups of four waves.  The tile is TH x TW <= 256 output
// pixels (8 MFMA row tiles) by NP >= NO output channels (NP / 32 column
// tiles); wave w of a group owns row tiles 2w and 2w+1 and every column
// tile.  With 64 columns (KG = 1) the four waves, one per SIMD, each run
// every 16-deep slice of the reduction (taps x 64 channels) and write their
// own rows: four fragment reads per four MFMAs.  With 32 columns (KG = 2,
// the stem's 16-tap input gradient) that would be three reads per two MFMAs,
// so group g takes the slices g, g+2, ... instead (two waves per SIMD, one
// fragment per MFMA), group 1 adds its sums into group 0's through LDS, and
// group 0 writes the tile.  Pixels past TH x TW, past the image or past NO
// channels are computed on zeros or clamped rows and never stored.
struct HaloArgs {
    const bf16 *in, *filt, *bias;
    bf16 *out;
    int H, W, P, Q;              // input and output extents
    int R, S, ph, pw;            // taps, zero padding
    int NO, flip;                // output channels stored; flipped taps
    int TH, TW, tiles_w, tiles_img, tiles;
    int hr, hs, lor, los;        // output phases: halo taps (rows, columns) and the halo origin's offset
    uint32_t in_bytes, filt_bytes, out_bytes;
};

// Halo pixels per buffer: 320 of 64 channels (40 KB), 640 of 16 (20 KB, the
// least that holds the epilogue's staging).
template <int CH> constexpr int halo_max_px() { return CH == 64 ? 320 : 640; }
// ... and for the output phases of a stride-2 input gradient, whose
// epilogues stage in an LDS area of their own (264 pixels, 33 KB)
constexpr int halo_max_px_oph() { return 264; }

// Chunk swizzle of a pixel row of CH channels in LDS: 128-byte rows as the
// GEMM's k-contiguous tiles (swz_k); 32-byte rows (two 16-byte chunks) swap
// their chunks every 4 rows, so the 8 rows one 16-byte read reaches at a time
// cover all 32 banks.
template <int CH> __device__ __forceinline__ int halo_swz(int row) {
    if constexpr (CH == 64) return swz_k(row);
    else return (row >> 2) & 1;
}

// ST = 2: a stride-2 forward as the sum of its four stride phases.  Phase
// (a, b) takes the taps r = a, a + 2, ... and s = b, b + 2, ...; their input
// pixels (ST y + r - ph, ST x + s - pw) are the phase image
// (ST (y + r') + a - ph, ST (x + s') + b - pw), r = 2 r' + a, read at
// stride 2, on which the phase is a stride-1 correlation with r' and s'.
// A tile is then four work items, one halo each ((TH + R2 - 1) x
// (TW + S2 - 1) pixels of the phase image, R2 = ceil(R / 2), the same shape
// for every phase so that the lanes' load offsets are worked out once),
// whose sums accumulate before the one epilogue; the phases of a tile
// reread neighbouring pixels of the same lines, mostly from L2.
//
// OPH: the input gradient of a stride-2 convolution as its four output
// phases.  Output pixel (2 i + a, 2 j + b) of dx takes the taps
// r = r0 + 2 u (r0 = (a + ph) mod 2) and s = s0 + 2 v, which read dy at
// (i + e_a - u, j + e_b - v), e_a = (a + ph - r0) / 2: each phase is a
// stride-1 correlation of dy on the phase image (i, j).  All four read the
// same dy neighbourhood, so a tile of the phase image is one halo (origin
// (i0 + lor, j0 + los), (TH + hr - 1) x (TW + hs - 1) pixels) and four work
// items, each with its own taps and epilogue (output rows and columns 2
// apart).  The epilogues stage in an LDS area of their own, so the halo
// stays for the next phase; the halo buffers are smaller to make room.
// (Stores straight from the accumulators, 8 bytes per lane, would free that
// area, but each one touches 32 pixel lines: 57 against 54 us.)
template <int NP, int TAPS_MAX, int KG, bool EXACT = false, int CH = 64, int ST = 1, bool OPH = false>
__global__ __launch_bounds__(KG * 256, 1) void halo_conv_kernel(const HaloArgs A) {
    static_assert(CH == 64 || (CH == 16 && KG == 1 && EXACT), "16-channel pixels: one group, exact taps");
    static_assert(ST == 1 || (ST == 2 && KG == 1 && !EXACT && CH == 64), "stride 2: one group, generic taps");
    static_assert(!OPH || (ST == 1 && KG == 1 && !EXACT && CH == 64), "output phases: one group, generic taps");
    constexpr int NPH = OPH ? 4 : ST * ST;          // work items (stride phases) per tile
    constexpr int NW = 4 * KG;                      // waves: KG k-groups of four
    constexpr int PB = CH * 2;                      // bytes of a pixel (or filter) row
    constexpr int CPR = CH / 8;                     // 16-byte chunks per row
    constexpr int RPI = 64 / CPR;                   // rows per LDS-DMA instruction
    constexpr int MAXPX = OPH ? halo_max_px_oph() : halo_max_px<CH>();
    constexpr int FILT_BYTES = TAPS_MAX * NP * PB;
    constexpr int HALO_BYTES = MAXPX * PB;
    constexpr int TN = NP / 32;
    constexpr int TM = 2;                           // row tiles per wave
    constexpr int EPI_PITCH = NP + 8;               // staged row, bf16 elements
    constexpr int STAGE_BYTES = OPH ? 4 * 32 * EPI_PITCH * 2 : 0;   // the output phases' own staging
    static_assert(FILT_BYTES + 2 * HALO_BYTES + STAGE_BYTES <= 160 * 1024, "LDS");
    static_assert(OPH || 4 * 32 * EPI_PITCH * 2 <= HALO_BYTES, "epilogue staging fits a halo buffer");
    static_assert(KG == 1 || 4 * TN * 16 * 64 * 4 <= HALO_BYTES, "one row tile of group 1's sums fits a halo buffer");
    __shared__ __attribute__((aligned(1024))) char smem[FILT_BYTES + 2 * HALO_BYTES + STAGE_BYTES];
    char *const sF = smem;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int kg = KG == 2 ? wave >> 2 : 0, wl = wave & 3;   // k-group, wave within it
    const int taps = A.R * A.S;
    // halo taps: per input phase at most (ST = 2), or the output phases' span (OPH)
    const int R2 = OPH ? A.hr : (A.R + ST - 1) / ST, S2 = OPH ? A.hs : (A.S + ST - 1) / ST;
    const int HWW = A.TW + S2 - 1;                    // halo row length
    const int HP = (A.TH + R2 - 1) * HWW;             // halo pixels
    const __amdgpu_buffer_rsrc_t rin = rsrc(A.in, A.in_bytes);
    const __amdgpu_buffer_rsrc_t rf = rsrc(A.filt, A.filt_bytes);
    const __amdgpu_buffer_rsrc_t ro = rsrc(A.out, A.out_bytes);
    // the lane's 16-byte slot of a row, and the logical k chunk it holds in
    // row `row`
    const int slot = lane % CPR;
    auto chunk_of = [&](int row) { return slot ^ halo_swz<CH>(row); };
    // fragment of row `row`: chunk pair `sub`, this lane's half
    auto frag = [&](const char *base, int row, int sub) {
        const int chunk = 2 * sub + (lane >> 5);
        return *reinterpret_cast<const bf16x8 *>(base + row * PB + ((chunk ^ halo_swz<CH>(row)) << 4));
    };

    // bias of the lane's output columns (added in fp32 before the rounding):
    // 4 consecutive channels per load through a descriptor of NO entries
    // (none without a bias), so columns past NO read zeros and every load is
    // in flight at once
    const int fr = lane & 31, fh = lane >> 5;
    float bcol[TN][4][4];
    {
        const __amdgpu_buffer_rsrc_t rb = rsrc(A.bias, A.bias ? (uint32_t)A.NO * 2u : 0u);
        typedef unsigned v2u32 __attribute__((ext_vector_type(2)));
        v2u32 bv[TN][4];
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                bv[j][q] = __builtin_amdgcn_raw_buffer_load_b64(rb, (j * 32 + 8 * q + 4 * fh) * 2, 0, 0);
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const uint32_t w = bv[j][q][v >> 1];
                    bcol[j][q][v] = __uint_as_float((v & 1) ? (w & 0xffff0000u) : (w << 16));
                }
    }

    // ---- the filter, once: LDS row t * NP + n = output channel n at tap t
    {
        const int rows = taps * NP, ninstr = (rows + RPI - 1) / RPI;
        for (int j = wave; j < ninstr; j += NW) {
            const int L = j * RPI + lane / CPR;
            const int t = L / NP, n = L - t * NP;
            const int ts = A.flip ? taps - 1 - t : t;
            const bool ok = t < taps && n < A.NO;
            const uint32_t off = ok ? (uint32_t)((n * taps + ts) * CH + chunk_of(n) * 8) * 2u : kOOB;
            dma16<false>(rf, sF + j * 1024, off);
        }
    }
    // ---- the halo of tile `tile` into buffer `b`.  Load instruction
    // j = wave + NW jj carries halo pixels RPI j .. RPI j + RPI - 1, the same
    // ones for every tile: their rows, columns and element offsets within the
    // halo are worked out once (rows past the halo are sent out of range).
    constexpr int HJ = (MAXPX / RPI + NW - 1) / NW;
    const int ninstr = (HP + RPI - 1) / RPI;
    int h_y[HJ], h_x[HJ];
    uint32_t h_c[HJ];
#pragma unroll
    for (int jj = 0; jj < HJ; ++jj) {
        const int hp = (wave + jj * NW) * RPI + lane / CPR;
        const int hy = hp / HWW, hx = hp - hy * HWW;
        h_y[jj] = hp < HP ? hy : -(1 << 20);
        h_x[jj] = hx;
        h_c[jj] = ((uint32_t)(ST * hy) * (uint32_t)A.W + (uint32_t)(ST * hx)) * (uint32_t)CH +
                  (uint32_t)chunk_of(hp) * 8u;
    }
    // the halo of phase `ph2` (= 2a + b) of tile `tile`
    auto load_halo = [&](int tile, int ph2, int b) {
        char *dst = smem + FILT_BYTES + b * HALO_BYTES;
        const int img = tile / A.tiles_img, rem = tile - img * A.tiles_img;
        const int ty = rem / A.tiles_w, tx = rem - ty * A.tiles_w;
        const int iy0 = OPH ? ty * A.TH + A.lor : ST * ty * A.TH + (ph2 >> 1) - A.ph;
        const int ix0 = OPH ? tx * A.TW + A.los : ST * tx * A.TW + (ph2 & 1) - A.pw;
        const int gbase = ((img * A.H + iy0) * A.W + ix0) * CH;
#pragma unroll
        for (int jj = 0; jj < HJ; ++jj) {
            const int j = wave + jj * NW;
            if (j >= ninstr) break;
            const int iy = iy0 + ST * h_y[jj], ix = ix0 + ST * h_x[jj];
            const bool ok = (unsigned)iy < (unsigned)A.H && (unsigned)ix < (unsigned)A.W;
            // element index below 2^31 (operand_fits), byte offset below kOOB
            const uint32_t off = ok ? ((uint32_t)gbase + h_c[jj]) * 2u : kOOB;
            dma16<false>(rin, dst + j * 1024, off);
        }
    };

    // per-lane halo rows of the wave's row tiles (tap (0, 0))
    const int npx = A.TH * A.TW;
    int base[TM];
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        const int p = (TM * wl + i) * 32 + fr;
        const int pp = p < npx ? p : 0;
        const int oy = pp / A.TW;
        base[i] = oy * HWW + (pp - oy * A.TW);
    }
    // output stores per wave and tile: a fixed count (masked lanes store past
    // the output's buffer range, which the hardware drops), so the wait for a
    // halo can leave the previous tile's stores in flight
    constexpr int NPASS = NP / 16;                  // 32 rows x NP/8 pieces over 64 lanes
    constexpr int SEG = NP / 8;                     // 16-byte pieces of a staged pixel row
    // the output pixel (row, column within the tile) and element offset of
    // each of the lane's stores, the same for every tile
    int e_y[TM][NPASS], e_x[TM][NPASS], e_c[TM][NPASS];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int ps = 0; ps < NPASS; ++ps) {
            const int lin = ps * 64 + lane;
            const int rl = lin / SEG, cl = (lin % SEG) * 8;
            const int p = (TM * wl + i) * 32 + rl;
            const int oy = p / A.TW, ox = p - oy * A.TW;
            const bool ok = cl < A.NO && p < npx;
            e_y[i][ps] = ok ? oy : (1 << 20);
            e_x[i][ps] = ox;
            e_c[i][ps] = ((OPH ? 2 : 1) * oy * A.Q + (OPH ? 2 : 1) * ox) * A.NO + cl;
        }
    int tap_r[TAPS_MAX], tap_s[TAPS_MAX];           // (r, s) of tap t
#pragma unroll
    for (int t = 0; t < TAPS_MAX; ++t) {
        tap_r[t] = t / A.S;
        tap_s[t] = t - tap_r[t] * A.S;
    }
    // work item `it` of this block: phase it % NPH of its (it / NPH)-th tile
    int tile = blockIdx.x, ph2 = 0;
    if (tile < A.tiles) load_halo(tile, 0, 0);
    floatx16 acc[TM][TN];
    for (int it = 0; tile < A.tiles; ++it) {
        // one halo per work item, or per tile (OPH)
        const int b = OPH ? (it / NPH) & 1 : it & 1;
        const char *sH = smem + FILT_BYTES + b * HALO_BYTES;
        if (!OPH || ph2 == 0) {
            // this wave's loads of the filter and of this halo landed (group
            // 0's stores, issued after them by the previous tile's
            // epilogue(s), may still be in flight)
            if (it == 0 || kg == 1 || (!OPH && ph2 != 0)) wait_vmcnt<0>();
            else wait_vmcnt<(OPH ? NPH : 1) * TM * NPASS>();
            wait_lgkm0();
            block_sync<true>();     // every wave's loads landed; the other buffer is free
            // the next work item's (OPH: tile's) halo lands while this one computes
            const int nph = !OPH && ph2 + 1 < NPH ? ph2 + 1 : 0;
            const int ntile = !OPH && ph2 + 1 < NPH ? tile : tile + (int)gridDim.x;
            if (ntile < A.tiles) load_halo(ntile, nph, b ^ 1);
        }

        if (OPH || ph2 == 0) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
        }
        bf16x8 fa[3][TM], fb[3][TN];
        // fragments of one slice: the row tiles' halo rows at halo offset
        // (r, s) and the filter rows of tap t, chunk pair `sub`
        auto read = [&](int r, int s, int t, int sub, int buf) {
            const int shift = r * HWW + s;
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[buf][i] = frag(sH, base[i] + shift, sub);
            const char *sFt = sF + t * NP * PB;
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[buf][j] = frag(sFt, j * 32 + fr, sub);
        };
        auto mfma = [&](int buf) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[buf][j], fa[buf][i], acc[i][j], 0, 0, 0);
        };
        if constexpr (EXACT) {
            // exactly TAPS_MAX taps: every slice of the group (all four of
            // each tap, or slices kg and kg + 2 with two k-groups) unrolled,
            // fragments read two slices ahead, slice k in buffer k mod 3
            constexpr int SPT = CH / 16 / KG;       // slices per tap and group
            constexpr int NSL = SPT * TAPS_MAX;
            auto rd = [&](int k) {
                const int t = k / SPT, sub = KG == 1 ? k % SPT : kg + 2 * (k % SPT);
                read(tap_r[t], tap_s[t], t, sub, k % 3);
            };
            rd(0);
            rd(1);
#pragma unroll
            for (int k = 0; k < NSL; ++k) {
                if (k + 2 < NSL) rd(k + 2);
                mfma(k % 3);
            }
        } else {
            // group kg takes slices kg and kg + 2 of every tap (one group: all
            // four); the next slice's fragments are read while a slice's MFMAs
            // run.  The phase's taps are (a + ST r, b + ST s), r < nr, s < ns,
            // at halo offset (r, s) (stride 1: every tap, at (r, s)).
            // OPH: output phase (pa, pb)'s taps (r0 + 2 r, s0 + 2 s) at halo
            // offset (er - r - lor, es - s - los)
            const int pa = ph2 >> 1, pb = ph2 & 1;
            const int r0 = (pa + A.ph) & 1, s0 = (pb + A.pw) & 1;
            const int er = (pa + A.ph - r0) / 2 - A.lor, es = (pb + A.pw - s0) / 2 - A.los;
            const int nr = OPH ? (A.R - r0 + 1) / 2 : (A.R - pa + ST - 1) / ST;
            const int ns = OPH ? (A.S - s0 + 1) / 2 : (A.S - pb + ST - 1) / ST, nt = nr * ns;
            auto tap_of = [&](int r, int s) {
                return OPH ? (r0 + 2 * r) * A.S + s0 + 2 * s : (pa + ST * r) * A.S + pb + ST * s;
            };
            auto hr_of = [&](int r) { return OPH ? er - r : r; };   // halo offset of tap row r
            auto hs_of = [&](int s) { return OPH ? es - s : s; };
            read(hr_of(0), hs_of(0), tap_of(0, 0), kg, 0);
            for (int i = 0, r = 0, s = 0; i < nt; ++i) {
                int r1 = r, s1 = s + 1;                 // the next tap
                if (s1 == ns) {
                    s1 = 0;
                    ++r1;
                }
                const int t = tap_of(r, s), hr = hr_of(r), hs = hs_of(s);
                if constexpr (KG == 2) {
                    read(hr, hs, t, kg + 2, 1);
                    mfma(0);
                } else {
                    read(hr, hs, t, 1, 1);
                    mfma(0);
                    read(hr, hs, t, 2, 0);
                    mfma(1);
                    read(hr, hs, t, 3, 1);
                    mfma(0);
                }
                if (i + 1 < nt) read(hr_of(r1), hs_of(s1), tap_of(r1, s1), kg, 0);
                mfma(1);
                r = r1;
                s = s1;
            }
        }

        // ---- group 1's sums into group 0's, one row tile at a time, through
        // this tile's halo buffer (every wave is done reading it after the
        // first barrier)
        float *red = reinterpret_cast<float *>(smem + FILT_BYTES + b * HALO_BYTES);
#pragma unroll
        for (int i = 0; i < (KG == 2 ? TM : 0); ++i) {
            wait_lgkm0();
            block_sync<true>();
            if (kg == 1) {
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int v = 0; v < 16; ++v) red[((wl * TN + j) * 16 + v) * 64 + lane] = acc[i][j][v];
            }
            wait_lgkm0();
            block_sync<true>();
            if (kg == 0) {
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int v = 0; v < 16; ++v) acc[i][j][v] += red[((wl * TN + j) * 16 + v) * 64 + lane];
            }
        }
        // the next work item: the tile's next phase, or the block's next tile
        const int cur_tile = tile, cur_ph = ph2;
        if (++ph2 == NPH) {
            ph2 = 0;
            tile += gridDim.x;
        }
        if (!OPH && ph2 != 0) continue;   // the tile's sums are not complete yet
        if constexpr (!OPH) {
            wait_lgkm0();
            block_sync<true>();   // the halo (and the sums) are read before the staging reuses the buffer
        }
        if (kg == 1) continue;

        // ---- epilogue (group 0): stage 32 rows per wave in this tile's halo
        // buffer, 16-byte stores
        const int img = cur_tile / A.tiles_img, rem = cur_tile - img * A.tiles_img;
        const int ty0 = (rem / A.tiles_w) * A.TH, tx0 = (rem - (rem / A.tiles_w) * A.tiles_w) * A.TW;
        // OPH: output phase (oa, ob), rows and columns 2 apart
        constexpr int OS = OPH ? 2 : 1;
        const int oa = OPH ? cur_ph >> 1 : 0, ob = OPH ? cur_ph & 1 : 0;
        const int obase = ((img * A.P + OS * ty0 + oa) * A.Q + OS * tx0 + ob) * A.NO;
        typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
        // (OPH: in the staging area past the halo buffers, which the next phases still read)
        bf16 *stage = reinterpret_cast<bf16 *>(smem + FILT_BYTES + (OPH ? 2 : b) * HALO_BYTES) + wl * 32 * EPI_PITCH;
#pragma unroll
        for (int i = 0; i < TM; ++i) {
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    bf16x4 o;
#pragma unroll
                    for (int v = 0; v < 4; ++v) o[v] = (bf16)(acc[i][j][4 * q + v] + bcol[j][q][v]);
                    *reinterpret_cast<bf16x4 *>(stage + fr * EPI_PITCH + j * 32 + 8 * q + 4 * fh) = o;
                }
            wait_lgkm0();
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int ps = 0; ps < NPASS; ++ps) {
                const int lin = ps * 64 + lane;
                const int rl = lin / SEG, cl = (lin % SEG) * 8;
                const u32x4 v = *reinterpret_cast<const u32x4 *>(stage + rl * EPI_PITCH + cl);
                const bool ok = OS * (ty0 + e_y[i][ps]) + oa < A.P && OS * (tx0 + e_x[i][ps]) + ob < A.Q;
                // element index below 2^31 (operand_fits on the output)
                const uint32_t off = ok ? (uint32_t)(obase + e_c[i][ps]) * 2u : kOOB;
                __builtin_amdgcn_raw_buffer_store_b128(v, ro, (int)off, 0, 0);
            }
            wait_lgkm0();
            __builtin_amdgcn_wave_barrier();
        }
    }
    wait_vmcnt<0>();   // no load of this block is still writing LDS when it ends
}

// Wt[c][rs][k] = W[k][rs][c]: the input gradient reads the (frozen) filter
// with its reduction index k contiguous.  K and C are multiples of 8 (the
// input gradient's fast path pads C and refuses other K), so W splits into
// whole 8 (k) x 8 (c) blocks of one tap, and each thread moves one in
// registers: eight 16-byte row loads (all in flight together), the transpose
// by 16-bit halves, eight 16-byte stores.  The 16 lanes of a block row take
// adjacent c blocks (one 256-byte run of a W row per load), the 8 block rows
// adjacent k blocks (64-byte runs of a Wt row per store, merged in L2).  No
// LDS and no barrier: a block is 64 k x 128 c of one tap.
// Grid (ceil(C/128), ceil(K/64), R*S), 128 threads.
__global__ __launch_bounds__(128) void transpose_krsc_kernel(const bf16 *__restrict__ W, bf16 *__restrict__ Wt,
                                                             int K, int RS, int C) {
    const int cb = blockIdx.x * 16 + (threadIdx.x & 15);   // 8-column block
    const int kb = blockIdx.y * 8 + (threadIdx.x >> 4);    // 8-row block
    const int rs = blockIdx.z;
    if (cb * 8 >= C || kb * 8 >= K) return;
    u32x4 v[8];
#pragma unroll
    for (int r = 0; r < 8; ++r)
        v[r] = *reinterpret_cast<const u32x4 *>(W + ((size_t)(kb * 8 + r) * RS + rs) * C + cb * 8);
#pragma unroll
    for (int c = 0; c < 8; ++c) {
        // column c of the block: element c of rows 0..7, two per word
        u32x4 o;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const uint32_t lo = v[2 * q][c / 2], hi = v[2 * q + 1][c / 2];
            o[q] = (c & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
        }
        *reinterpret_cast<u32x4 *>(Wt + ((size_t)(cb * 8 + c) * RS + rs) * K + kb * 8) = o;
    }
}

int transpose_krsc(const void *w, bf16 *wt, int K, int RS, int C, hipStream_t st) {
    if (K % 8 != 0 || C % 8 != 0) return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(transpose_krsc_kernel, dim3((C + 127) / 128, (K + 63) / 64, RS), dim3(128), 0, st,
                       (const bf16 *)w, wt, K, RS, C);
    return (int)hipGetLastError();
}

// Channel counts that are not a multiple of 8 (the 3-channel stem): the fast
// path runs on copies whose channels are padded with zeros to C8 =
// roundup(C, 8).  dst[row][c] = c < C ? src[row][c] : 0, one 16-byte row
// vector per thread.
__global__ __launch_bounds__(256) void pad_channels_kernel(const bf16 *__restrict__ src, int64_t rows, int C, int C8,
                                                           bf16 *__restrict__ dst) {
    const int nv = C8 / 8;
    const int64_t total = rows * nv;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = i / nv;
        const int c0 = (int)(i - row * nv) * 8;
        Vec16<bf16> v;
#pragma unroll
        for (int e = 0; e < 8; ++e) v.e[e] = c0 + e < C ? src[row * C + c0 + e] : (bf16)0.f;
        store16(dst + row * C8 + c0, v);
    }
}

// Pair packing for narrow inputs with a stride-2 width (the 3-channel stem):
// each 8-channel pixel u of the packed input holds the columns 2u - pw and
// 2u + 1 - pw of up to 4 channels (zeros past C and outside the width), so the
// stride-2 convolution over W becomes a stride-1 convolution over pixel pairs
// with ceil(S / 2) taps and no width padding.
//   xq[row][u][4t + c] = x[row][2u + t - pw][c]        (row = (n, h))
//   wq[kr][j][4t + c]  = w[kr][2j + t][c]   (0 for 2j + t >= S)  (kr = (k, r))
__global__ __launch_bounds__(256) void pack_pairs_kernel(const bf16 *__restrict__ x, int64_t rows, int W, int C,
                                                         int Wq, int pw, bf16 *__restrict__ xq) {
    const int64_t total = rows * Wq;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = i / Wq;
        const int u = (int)(i - row * Wq);
        Vec16<bf16> v;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int c = e & 3, w = 2 * u + (e >> 2) - pw;
            v.e[e] = c < C && w >= 0 && w < W ? x[(row * W + w) * C + c] : (bf16)0.f;
        }
        store16(xq + i * 8, v);
    }
}

__global__ __launch_bounds__(256) void pack_pair_filter_kernel(const bf16 *__restrict__ w, int64_t KR, int S, int C,
                                                               int Sq, bf16 *__restrict__ wq) {
    const int64_t total = KR * Sq;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t kr = i / Sq;
        const int j = (int)(i - kr * Sq);
        Vec16<bf16> v;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const int c = e & 3, s = 2 * j + (e >> 2);
            v.e[e] = c < C && s < S ? w[(kr * S + s) * C + c] : (bf16)0.f;
        }
        store16(wq + i * 8, v);
    }
}

// the adjoints of the packings: dx[row][w][c] = dxq[row][(w + pw) / 2][4 ((w + pw) % 2) + c],
// dw[kr][s][c] = dwq[kr][s / 2][4 (s % 2) + c]
__global__ __launch_bounds__(256) void unpack_pairs_kernel(const bf16 *__restrict__ dxq, int64_t rows, int W, int C,
                                                           int Wq, int pw, bf16 *__restrict__ dx) {
    const int64_t total = rows * W * C;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t rw = i / C;
        const int c = (int)(i - rw * C);
        const int64_t row = rw / W;
        const int w = (int)(rw - row * W) + pw;
        dx[i] = dxq[(row * Wq + w / 2) * 8 + 4 * (w & 1) + c];
    }
}

__global__ __launch_bounds__(256) void unpack_pair_filter_kernel(const bf16 *__restrict__ dwq, int64_t KR, int S,
                                                                 int C, int Sq, bf16 *__restrict__ dw) {
    const int64_t total = KR * S * C;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t ks = i / C;
        const int c = (int)(i - ks * C);
        const int64_t kr = ks / S;
        const int s = (int)(ks - kr * S);
        dw[i] = dwq[(kr * Sq + s / 2) * 8 + 4 * (s & 1) + c];
    }
}

// 2 x 2 pixel blocks, for the input gradient of a layer with at most 4
// input channels and stride 2 in both dimensions: with the padded input cut
// into 2 x 2 blocks, xq[n][i][j][8a + 4b + c] = x[n][2i + a - ph][2j + b - pw][c],
// the layer is a stride-1 convolution of xq with the filter
// wq[k][r'][s'][8a + 4b + c] = w[k][2r' + a][2s' + b][c] (zeros past R, S, C).
// Its input gradient has 16 columns (pairs along W alone give 8 and two
// stride phases).  One thread writes the 16 channels of one (k, r', s').
__global__ __launch_bounds__(256) void pack_block_filter_kernel(const bf16 *__restrict__ w, int K, int R, int S, int C,
                                                                int Rq, int Sq, bf16 *__restrict__ wq) {
    const int64_t total = (int64_t)K * Rq * Sq;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t k = i / (Rq * Sq);
        const int rs = (int)(i - k * (Rq * Sq));
        const int rq = rs / Sq, sq = rs - rq * Sq;
        Vec16<bf16> v[2];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int a = e >> 3, b = (e >> 2) & 1, c = e & 3;
            const int r = 2 * rq + a, s = 2 * sq + b;
            v[e >> 3].e[e & 7] = c < C && r < R && s < S ? w[((k * R + r) * S + s) * C + c] : (bf16)0.f;
        }
        store16(wq + i * 16, v[0]);
        store16(wq + i * 16 + 8, v[1]);
    }
}

// the adjoint of the input packing:
// dx[n][h][w][c] = dxq[n][(h + ph) / 2][(w + pw) / 2][8 ((h + ph) % 2) + 4 ((w + pw) % 2) + c]
// One thread per (image row n, h; block column j): the 16-byte half of block
// (n, (h + ph) / 2, j) that holds row h carries both of its columns,
// w = 2j - pw and 2j + 1 - pw, so each output pixel is written exactly once.
// 32-bit indices: the host checks that the rows x block columns fit.
__global__ __launch_bounds__(256) void unpack_blocks_kernel(const bf16 *__restrict__ dxq, uint32_t NH, int H, int W,
                                                            int C, int Hq, int Wq, int ph, int pw,
                                                            bf16 *__restrict__ dx) {
    const uint32_t total = NH * (uint32_t)Wq;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        const uint32_t nh = i / (uint32_t)Wq, j = i - nh * (uint32_t)Wq;
        const uint32_t n = nh / (uint32_t)H, h = nh - n * (uint32_t)H;
        const uint32_t hp = h + (uint32_t)ph;
        const Vec16<bf16> v = load16(dxq + (((size_t)n * Hq + hp / 2) * Wq + j) * 16 + 8 * (hp & 1));
        bf16 *row = dx + (size_t)nh * W * C;
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int w = 2 * (int)j + b - pw;
            if (w < 0 || w >= W) continue;
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if (c < C) row[w * C + c] = v.e[4 * b + c];
        }
    }
}

// The same, with the row staged in LDS so that dx is written in 16-byte
// vectors: one workgroup per image row (n, h), rows of W * C elements a
// multiple of 8 (the host checks).  Thread j loads the half block that
// holds row h for block column j and puts its pixels' C channels in place
// in the LDS row; then the row leaves as ceil(W * C / 8) 16-byte stores.
constexpr int kUnpackRowMax = 2048;   // LDS row capacity in elements (4 KB)
__global__ __launch_bounds__(256) void unpack_blocks_row_kernel(const bf16 *__restrict__ dxq, int H, int W, int C,
                                                                int Hq, int Wq, int ph, int pw,
                                                                bf16 *__restrict__ dx) {
    __shared__ __attribute__((aligned(16))) bf16 row[kUnpackRowMax];
    const uint32_t nh = blockIdx.x, n = nh / (uint32_t)H, h = nh - n * (uint32_t)H;
    const uint32_t hp = h + (uint32_t)ph;
    const bf16 *src = dxq + (((size_t)n * Hq + hp / 2) * Wq) * 16 + 8 * (hp & 1);
    for (int j = threadIdx.x; j < Wq; j += blockDim.x) {
        const Vec16<bf16> v = load16(src + (size_t)j * 16);
#pragma unroll
        for (int b = 0; b < 2; ++b) {
            const int w = 2 * j + b - pw;
            if (w < 0 || w >= W) continue;
#pragma unroll
            for (int c = 0; c < 4; ++c)
                if (c < C) row[w * C + c] = v.e[4 * b + c];
        }
    }
    __syncthreads();
    const int nv = W * C / 8;
    u32x4 *out = reinterpret_cast<u32x4 *>(dx + (size_t)nh * W * C);
    for (int k = threadIdx.x; k < nv; k += blockDim.x) out[k] = reinterpret_cast<const u32x4 *>(row)[k];
}

// The forward's input in 2 x 2 pixel blocks (at most 4 channels, stride 2
// in both dimensions): xq[n][i][j][8a + 4b + c] = x[n][2i + a - ph][2j + b - pw][c],
// zeros outside the image and for c >= C.  One thread writes the 16 channels
// of one block; its reads go through the buffer descriptor of x, positions
// outside sent past its range, so all 16 are issued at once.  32-bit
// indices: the host checks that the blocks and x fit.
__global__ __launch_bounds__(256) void pack_blocks_kernel(const bf16 *__restrict__ x, uint32_t N, int H, int W, int C,
                                                          int Hq, int Wq, int ph, int pw, bf16 *__restrict__ xq) {
    const __amdgpu_buffer_rsrc_t rx = rsrc(x, (uint32_t)N * (uint32_t)H * (uint32_t)W * (uint32_t)C * 2u);
    const uint32_t total = N * (uint32_t)Hq * (uint32_t)Wq;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        const uint32_t ni = i / (uint32_t)Wq, j = i - ni * (uint32_t)Wq;
        const uint32_t n = ni / (uint32_t)Hq, iq = ni - n * (uint32_t)Hq;
        unsigned short u[16];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int a = e >> 3, b = (e >> 2) & 1, c = e & 3;
            const int h = 2 * (int)iq + a - ph, w = 2 * (int)j + b - pw;
            const bool ok = c < C && (unsigned)h < (unsigned)H && (unsigned)w < (unsigned)W;
            const uint32_t off = ok ? (((n * (uint32_t)H + (uint32_t)h) * (uint32_t)W + (uint32_t)w) * (uint32_t)C + c) * 2u : kOOB;
            u[e] = __builtin_amdgcn_raw_buffer_load_b16(rx, (int)off, 0, 0);
        }
        u32x4 v0, v1;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            v0[q] = (uint32_t)u[2 * q] | ((uint32_t)u[2 * q + 1] << 16);
            v1[q] = (uint32_t)u[8 + 2 * q] | ((uint32_t)u[8 + 2 * q + 1] << 16);
        }
        *reinterpret_cast<u32x4 *>(xq + (size_t)i * 16) = v0;
        *reinterpret_cast<u32x4 *>(xq + (size_t)i * 16 + 8) = v1;
    }
}

// The same, with the two input rows of a block row staged in LDS so that x
// is read in 16-byte vectors: one workgroup per block row (n, i), rows of
// W * C elements a multiple of 8 (the host checks).  Rows 2i - ph and
// 2i + 1 - ph land in LDS (zeros outside the image); thread j then gathers
// block (n, i, j) from LDS and writes its 16 channels as two 16-byte stores.
__global__ __launch_bounds__(256) void pack_blocks_row_kernel(const bf16 *__restrict__ x, int H, int W, int C, int Hq,
                                                              int Wq, int ph, int pw, bf16 *__restrict__ xq) {
    __shared__ __attribute__((aligned(16))) bf16 rows[2][kUnpackRowMax];
    const uint32_t ni = blockIdx.x, n = ni / (uint32_t)Hq, iq = ni - n * (uint32_t)Hq;
    const int nv = W * C / 8;
#pragma unroll
    for (int a = 0; a < 2; ++a) {
        const int h = 2 * (int)iq + a - ph;
        const bool in = (unsigned)h < (unsigned)H;
        const u32x4 *src = reinterpret_cast<const u32x4 *>(x + ((size_t)n * H + (in ? h : 0)) * W * C);
        for (int k = threadIdx.x; k < nv; k += blockDim.x)
            reinterpret_cast<u32x4 *>(rows[a])[k] = in ? src[k] : u32x4{0u, 0u, 0u, 0u};
    }
    __syncthreads();
    for (int j = threadIdx.x; j < Wq; j += blockDim.x) {
        Vec16<bf16> v[2];
#pragma unroll
        for (int e = 0; e < 16; ++e) {
            const int a = e >> 3, b = (e >> 2) & 1, c = e & 3;
            const int w = 2 * j + b - pw;
            v[e >> 3].e[e & 7] = c < C && (unsigned)w < (unsigned)W ? rows[a][w * C + c] : (bf16)0.f;
        }
        bf16 *dst = xq + ((size_t)ni * Wq + j) * 16;
        store16(dst, v[0]);
        store16(dst + 8, v[1]);
    }
}

// dst[row][c] = src[row][c] for c < C (drops the padding channels).
__global__ __launch_bounds__(256) void crop_channels_kernel(const bf16 *__restrict__ src, int64_t rows, int C8, int C,
                                                            bf16 *__restrict__ dst) {
    const int64_t total = rows * C;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = i / C;
        const int c = (int)(i - row * C);
        dst[i] = src[row * C8 + c];
    }
}

// Sum split-K partials (and fused bias-gradient partials) to bf16; with a
// bias, out[i] also gets bias[i % ncol] (added in fp32 before the rounding).
__global__ __launch_bounds__(256) void reduce_kernel(const float *__restrict__ part, int splits, int64_t n,
                                                     int64_t pstride, bf16 *__restrict__ out, const float *__restrict__ dbpart,
                                                     int M, bf16 *__restrict__ db, const bf16 *__restrict__ bias,
                                                     int ncol) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t nv = n / 4;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nv; i += stride) {
        floatx4 s = *reinterpret_cast<const floatx4 *>(part + 4 * i);
        for (int z = 1; z < splits; ++z) s += *reinterpret_cast<const floatx4 *>(part + (int64_t)z * pstride + 4 * i);
        if (bias) {
#pragma unroll
            for (int e = 0; e < 4; ++e) s[e] += (float)bias[(4 * i + e) % ncol];
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) out[4 * i + e] = (bf16)s[e];
    }
    for (int64_t i = 4 * nv + (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride) {
        float s = 0.f;
        for (int z = 0; z < splits; ++z) s += part[(int64_t)z * pstride + i];
        if (bias) s += (float)bias[i % ncol];
        out[i] = (bf16)s;
    }
    if (dbpart) {
        for (int64_t m = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; m < M; m += stride) {
            float s = 0.f;
            for (int z = 0; z < splits; ++z) s += dbpart[(int64_t)z * M + m];
            db[m] = (bf16)s;
        }
    }
}

}  // namespace g2
}  // namespace ms

// ------------------------------------------------------------------ launchers
namespace ms {
namespace g2 {
namespace {

constexpr int kCUs = 256;

struct Tile {
    const char *name;
    int bm, bn;       // block tile
    int wr, wc;       // wave grid (wr * wc waves of (bm/wr) x (bn/wc))
    int stages;       // LDS ring depth (BK = 64 per stage)
    int per_cu;       // blocks resident per CU
    float eff1;       // relative MFMA efficiency with one block on the CU
    float eff;        // ... with per_cu blocks on the CU
    int kg = 1;       // k-groups of wr x wc waves (the block has wr * wc * kg waves)
};
// Efficiencies measured on the Linear and encoder shapes: a 2-stage
// 128 x 128 block alone on a CU cannot hide its load latency (a co-resident
// block normally does), where the 4-stage variant can.
constexpr Tile kTiles[] = {
    {"256x256", 256, 256, 2, 4, 2, 1, 1.20f, 1.20f},      // 8 waves of 128 x 64, 128 KB LDS
    {"256x128", 256, 128, 2, 4, 3, 1, 1.00f, 1.00f},      // 8 waves of 128 x 32, 144 KB
    {"128x128", 128, 128, 2, 2, 2, 2, 0.78f, 1.00f},      // 4 waves of 64 x 64, 64 KB, two blocks per CU
    {"128x128w8", 128, 128, 2, 4, 2, 2, 0.85f, 1.02f},    // 8 waves of 64 x 32, 64 KB, two blocks per CU
    {"128x128s4", 128, 128, 2, 2, 4, 1, 0.90f, 0.90f},    // 4 waves of 64 x 64, 4 stages (128 KB)
    {"128x128w8s4", 128, 128, 2, 4, 4, 1, 0.90f, 0.90f},  // 8 waves of 64 x 32, 4 stages (128 KB)
    {"128x128k2", 128, 128, 2, 2, 4, 1, 0.95f, 0.95f, 2},  // 2 k-groups of 4 waves of 64 x 64, 4 stages
    {"128x64", 128, 64, 2, 2, 2, 3, 0.75f, 0.75f},        // 4 waves of 64 x 32, 48 KB, three blocks per CU
    {"256x32", 256, 32, 4, 1, 2, 2, 0.70f, 0.70f},        // 4 waves of 64 x 32, 72 KB, two blocks per CU
    {"128x192k2", 128, 192, 2, 2, 3, 1, 0.82f, 0.82f, 2},  // 2 k-groups of 4 waves of 64 x 96, 3 stages (120 KB)
    {"256x288", 256, 288, 4, 3, 2, 1, 1.10f, 1.10f},      // 12 waves of 64 x 96, 2 stages (137 KB)
};
constexpr int kNumTiles = (int)(sizeof(kTiles) / sizeof(kTiles[0]));
// tiles the planner chooses from
// tiles the planner chooses from: the 4-wave 4-stage tile is kept for the
// tests; its 8-wave twin was as fast or faster on every measured shape
// (weight gradient 4096 x 1024 x 4096: 57 -> 46 us), and the k-group tile
// beats that one by ~5% on the forward and input gradient of 4096 x 1024
// outputs with K = 4096 (38.7 -> 36.3 us)
constexpr bool kAuto[kNumTiles] = {true, true, true, true, false, true, true, true, false, false, false};
// the narrow 256 x 32 tile is for thin outputs (N <= 32, e.g. the input
// gradient of a 3-channel image) and exists only for the contractions whose
// operands are both k-contiguous (forward, input gradient through the
// transposed filter): the transposing reads' swizzle assumes rows of at
// least 8 slots
constexpr bool narrow_tile(const Tile &t) { return t.bn < 64; }
// The 128 x 192 tile (two k-groups) also exists only for those contractions:
// its block width is not a power of two.  On 8192-row outputs it makes every
// encoder shape a whole number of waves (8192 x 768: 256 tiles, where
// 256 x 128 leaves 64 CUs idle).
constexpr bool kc_only(const Tile &t) { return narrow_tile(t) || t.bn == 192 || t.bn == 288; }
constexpr bool kAutoKc[kNumTiles] = {true, true, true, true, false, true, true, true, true, true, false};
// The 256 x 288 tile (12 waves of 64 x 96, three per SIMD) exists for the
// Linear forward only (the unit-geometry loads; the input gradient's fused
// bias column sums leave it short of registers).  An 8192 x 2304 output (the
// encoder's QKV forward) is 256 of its tiles, one wave, where 256 x 256
// makes 288 tiles: one wave plus a column-split remainder that runs on half
// the chip.
constexpr bool kAutoUnitKc[kNumTiles] = {true, true, true, true, false, true, true, true, true, true, true};
// tiles the planner chooses from for the input gradient of convolutions
// that are not 1x1 / stride 1 (implicit-GEMM gathers): on the
// ResNet-18-shaped stack's layers and the conv sweep the 2-stage 128 x 128
// tile (128 x 64 for 64 channels) was fastest or within 2% of it, and the
// 8-wave, 4-stage and k-group tiles lost by up to 35% (14 x 14 x 256: k-group
// 45 us against 33); that input gradient goes through the transposed filter
// (the in-place variant wants an 8-wave tile).  Whole steps on one box: the
// input-variant stack 2.32 -> 2.27 ms, the 3x3 conv sweep (input mask)
// 0.121 -> 0.116 ms.  The forward keeps the general set: restricted the same
// way it took split reductions whose extra pass made the frozen stack 6%
// slower.
constexpr bool kAutoConv[kNumTiles] = {true, false, true, false, false, false, false, true, true, false, false};
// tiles for convolutions on the tap-step operand loads (the forward with C,
// or the input gradient with K, a multiple of BK): without the per-lane
// divisions the 8-wave 4-stage 128 x 128 tile is the fastest or near it on
// the ResNet-18-shaped layers and the conv sweep (stage-3 input gradient 36.4
// -> 25.5 us against the 4-wave tile, stride-2 stage-4 31.2 -> 22.2 us,
// stage-3 forward 23.9 -> 20.9 us against the k-group tile), and the k-group
// tiles lose to it
constexpr bool kAutoTs[kNumTiles] = {true, true, true, true, false, true, false, true, true, false, false};

// MEMSAVE_GEMM_TILE=<name> forces one tile shape (a debugging and testing
// knob); returns its index or -1.
int forced_tile() {
    const char *e = getenv("MEMSAVE_GEMM_TILE");
    if (!e || !*e) return -1;
    for (int i = 0; i < kNumTiles; ++i)
        if (strcmp(kTiles[i].name, e) == 0) return i;
    return -1;
}

// ---------------------------------------------------------------- planner
// Estimated run time (microseconds) of a GEMM of M x N x K (z independent
// GEMMs of that bound, the stride phases of an input gradient) on tile t
// with the reduction split `splits` ways.  Per BK step a block takes the
// longer of its MFMA time (shared with the blocks resident on its CU) and
// the load latency its LDS ring can hide (STAGES - 1 tiles in flight); a
// wave of blocks also pays a fixed start/drain cost, every output byte is
// written once (fp32 partials when split), and a split adds the reduce pass.
// Constants come from kernel traces of the Linear and conv workloads: a
// 256 x 256 x 64 step of the 8-wave tile takes 1.5 us, a load round trip
// about 1 us.
constexpr double kUnitsPerUs = 2.33e6;   // bm*bn*k per us at relative efficiency 1
constexpr double kLoadUs = 1.0;          // HBM/L2 round trip of a stage's loads
constexpr double kWaveUs = 5.0;          // start + epilogue + drain of one wave of blocks
constexpr double kBytesPerUs = 6.0e6;    // streamed HBM bytes per us
constexpr double kLaunchUs = 3.0;

double est_us(const Tile &t, long M, long N, long K, int z, int splits) {
    const long tiles = ((M + t.bm - 1) / t.bm) * ((N + t.bn - 1) / t.bn) * z;
    const long blocks = tiles * splits;
    const long conc = (long)kCUs * t.per_cu;
    const long waves = (blocks + conc - 1) / conc;
    const long resident = std::min<long>(t.per_cu, (blocks + kCUs - 1) / kCUs);
    const long kper = ((K + splits - 1) / splits + BK - 1) / BK * BK;
    const double eff = resident > 1 ? t.eff : t.eff1;
    const double t_mfma = (double)resident * t.bm * t.bn * BK / (kUnitsPerUs * eff);
    const double t_lat = kLoadUs / (t.stages - 1);
    const double step = std::max(t_mfma, t_lat);
    const double out_elems = (double)M * N * z;
    double us = waves * ((double)(kper / BK) * step + kWaveUs) + out_elems * (splits > 1 ? 4.0 * splits : 2.0) / kBytesPerUs;
    if (splits > 1) us += kLaunchUs + out_elems * (4.0 * splits + 2.0) / kBytesPerUs;
    return us;
}

// MEMSAVE_GEMM_SPLITS=<n> forces the split count of the forward and
// input-gradient contractions (a testing knob, like MEMSAVE_GEMM_TILE).
int forced_splits() {
    const char *e = getenv("MEMSAVE_GEMM_SPLITS");
    if (!e || !*e) return 0;
    const int v = atoi(e);
    return v >= 1 ? std::min(v, 64) : 0;
}

struct GemmPlan {
    Tile t;
    int splits, k_split;
};

// Use of the k-group tile: by the planner, only when forced by the testing
// knob, or never (the weight gradient has no k-group instantiation).
enum KgUse { kKgNever = 0, kKgForced = 1, kKgAuto = 2 };

// Tile and split count for the forward or weight gradient (z = 1) or the input gradient (z stride
// phases) with at most max_splits splits of at least 4 BK steps each.
GemmPlan plan_gemm(long M, long N, long K, int z, int split_cap = 16, bool allow_256x256 = true,
                   int kgroups = kKgAuto, const bool *auto_set = kAuto) {
    int forced = forced_tile();
    // not built for the weight gradient: plan as usual
    if (forced >= 0 && (kTiles[forced].kg > 1 || kc_only(kTiles[forced])) && kgroups == kKgNever) forced = -1;
    // the in-place input gradient (its set is kAuto) has no k-contiguous-only tile: plan as usual
    if (forced >= 0 && kc_only(kTiles[forced]) && auto_set == kAuto) forced = -1;
    // the 288-wide tile exists for the unit-geometry forward only (its set is kAutoUnitKc)
    if (forced >= 0 && kTiles[forced].bn == 288 && auto_set != kAutoUnitKc) forced = -1;
    if (forced == 0 && !allow_256x256) forced = 1;   // the next widest tile (256 x 128)
    const int fs = split_cap > 1 ? forced_splits() : 0;
    const int max_splits = (int)std::max<long>(1, std::min<long>(split_cap, K / (4 * BK)));
    double best = 1e300;
    GemmPlan bp{kTiles[0], 1, (int)K};
    for (int ti = 0; ti < kNumTiles; ++ti) {
        if (forced >= 0 ? ti != forced : !auto_set[ti]) continue;
        if (ti == 0 && !allow_256x256) continue;
        if (kTiles[ti].kg > 1 && (kgroups == kKgNever || (kgroups == kKgForced && forced < 0))) continue;
        // the 192- and 288-wide tiles pay off only where they fill the CUs in
        // one wave (encoder shapes, 8192 x {768, 2304, 3072} outputs: 34
        // against 38 us at K = 2304 in one wave, 49 against 44 us in three
        // waves at K = 768)
        if (forced < 0 && (kTiles[ti].bn == 192 || kTiles[ti].bn == 288) &&
            ((M + kTiles[ti].bm - 1) / kTiles[ti].bm) * ((N + kTiles[ti].bn - 1) / kTiles[ti].bn) * z >
                (long)kCUs * kTiles[ti].per_cu)
            continue;
        for (int sp = 1; sp <= (fs ? 1 : max_splits); ++sp) {
            const int splits = fs ? fs : sp;
            const double us = est_us(kTiles[ti], M, N, K, z, splits);
            if (us < best * 0.999) {
                best = us;
                bp.t = kTiles[ti];
                bp.splits = splits;
            }
        }
    }
    long k_split = (K + bp.splits - 1) / bp.splits;
    k_split = std::max<long>(BK, (k_split + BK - 1) / BK * BK);
    bp.k_split = (int)k_split;
    bp.splits = K > 0 ? (int)((K + k_split - 1) / k_split) : 1;
    if (fs) bp.splits = fs;   // forced: keep the count even if some splits are empty
    return bp;
}

// Column split of a one-split, unit-geometry contraction whose tiles leave
// its last wave of blocks partly empty (an 8192 x 3072 output is 384 tiles
// of 256 x 256: one and a half waves of 256 CUs, so the second wave runs at
// half occupancy for as long as the first).  The first launch takes the
// leading n1 columns, as many whole tile columns as fit in the waves the
// plan's tiles fill completely; the second covers the remaining columns with
// the tile the planner
// picks for that narrower output (8192 x 1024: 256 tiles of 256 x 128).  The
// two launches write disjoint column ranges of one output (row stride = the
// full width) and neither needs workspace.  The split is taken when the
// estimate of the two launches plus the gap between them beats the one.
// MEMSAVE_GEMM_TAIL=off disables it and =on takes it wherever it applies
// (testing knobs).
struct ColSplit {
    int n1 = 0;     // columns of the first launch (0: no split)
    GemmPlan p2{};  // plan of the remaining columns
};
constexpr double kGapUs = 1.5;   // dispatch gap between two launches on one stream

int tail_mode() {
    const char *e = getenv("MEMSAVE_GEMM_TAIL");
    if (!e || !*e) return 1;
    if (strcmp(e, "off") == 0) return 0;
    if (strcmp(e, "on") == 0) return 2;
    return 1;
}

ColSplit col_split(const GemmPlan &p, long M, long N, long K, const bool *set) {
    ColSplit cs;
    const int mode = tail_mode();
    if (mode == 0 || p.splits != 1 || forced_tile() >= 0) return cs;
    const long ntm = (M + p.t.bm - 1) / p.t.bm, ntn = (N + p.t.bn - 1) / p.t.bn;
    const long conc = (long)kCUs * p.t.per_cu, tiles = ntm * ntn;
    if (tiles <= conc || tiles % conc == 0 || ntm > conc) return cs;
    const long c1 = (tiles / conc) * conc / ntm;   // tile columns of the whole waves
    if (c1 < 1 || c1 >= ntn) return cs;
    const long n1 = c1 * p.t.bn;
    const GemmPlan p2 = plan_gemm(M, N - n1, K, 1, 1, true, kKgAuto, set);
    const double one = est_us(p.t, M, N, K, 1, 1);
    const double two = est_us(p.t, M, n1, K, 1, 1) + est_us(p2.t, M, N - n1, K, 1, 1) + kGapUs;
    if (mode == 1 && two >= one) return cs;
    cs.n1 = (int)n1;
    cs.p2 = p2;
    return cs;
}

// floats of one split's partials (a multiple of 4: 16-byte aligned splits)
int64_t part_stride(int64_t elems) { return (elems + 3) / 4 * 4; }

// The launch records the profiling events itself when its kind is armed, so
// a pair spans this kernel's execution alone.
template <int MODE, int BM, int BN, int WR, int WC, int STAGES, int OCC, bool UNIT, int KG = 1, bool TS = false>
int go(const Args &a, dim3 grid, hipStream_t st) {
    const unsigned pk = MODE == kFwd ? kProfFwd : MODE == kWgrad ? kProfWgrad : kProfDgrad;
    void *eb = nullptr, *ee = nullptr;
    const bool timed = prof_pair(pk, &eb, &ee);
    hipExtLaunchKernelGGL((gemm_kernel<MODE, BM, BN, WR, WC, STAGES, OCC, UNIT, KG, TS>), grid,
                          dim3(WR * WC * KG * 64), 0, st, (hipEvent_t)eb, (hipEvent_t)ee, 0, a);
    const int err = (int)hipGetLastError();
    if (timed) prof_pair_done(pk, eb, ee, err == 0);
    return err;
}

// The strided input gradient has no 256 x 256 instantiation (its pixel
// mapping leaves that tile short of registers); the planner never picks it.
template <int MODE, bool UNIT>
constexpr bool has_256x256() { return !(MODE == kDgrad && !UNIT); }

template <int MODE, bool UNIT, bool TS = false>
int go_tile(const Tile &t, const Args &a, dim3 grid, hipStream_t st) {
    if (t.bn == 288) {
        if constexpr (MODE == kFwd && UNIT && !TS) return go<MODE, 256, 288, 4, 3, 2, 1, UNIT>(a, grid, st);
        else return (int)hipErrorInvalidValue;
    }
    if (t.bm == 256 && t.bn == 256) {
        // the weight gradient's 256 x 256 tile has no registers left for the
        // pixel cursor (it spilled): the generic loads
        constexpr bool TS2 = TS && MODE != kWgrad;
        if constexpr (has_256x256<MODE, UNIT>()) return go<MODE, 256, 256, 2, 4, 2, 1, UNIT, 1, TS2>(a, grid, st);
        else return (int)hipErrorInvalidValue;
    }
    if (t.bm == 256 && t.bn == 128) return go<MODE, 256, 128, 2, 4, 3, 1, UNIT, 1, TS>(a, grid, st);
    if (t.kg == 2) {
        if constexpr (MODE != kWgrad) {
            if (t.bm == 128 && t.bn == 128) return go<MODE, 128, 128, 2, 2, 4, 1, UNIT, 2, TS>(a, grid, st);
        }
        if constexpr (MODE == kFwd || MODE == kDgrad) {
            if (t.bm == 128 && t.bn == 192) return go<MODE, 128, 192, 2, 2, 3, 1, UNIT, 2, TS>(a, grid, st);
        }
        return (int)hipErrorInvalidValue;
    }
    if (t.bn == 32) {
        if constexpr (MODE == kFwd || MODE == kDgrad) return go<MODE, 256, 32, 4, 1, 2, 2, UNIT, 1, TS>(a, grid, st);
        return (int)hipErrorInvalidValue;
    }
    if (t.bm == 128 && t.bn == 128 && t.wc == 4 && t.stages == 4) return go<MODE, 128, 128, 2, 4, 4, 1, UNIT, 1, TS>(a, grid, st);
    if (t.bm == 128 && t.bn == 128 && t.wc == 4) return go<MODE, 128, 128, 2, 4, 2, 2, UNIT, 1, TS>(a, grid, st);
    if (t.bm == 128 && t.bn == 128 && t.stages == 4) return go<MODE, 128, 128, 2, 2, 4, 1, UNIT, 1, TS>(a, grid, st);
    if (t.bm == 128 && t.bn == 128) return go<MODE, 128, 128, 2, 2, 2, 2, UNIT, 1, TS>(a, grid, st);
    return go<MODE, 128, 64, 2, 2, 2, 3, UNIT, 1, TS>(a, grid, st);
}

// ts: a convolution forward, or input gradient through the transposed
// filter, whose steps each lie in one tap (channels of the reduction a
// multiple of BK, at most 32 taps per stride phase): the tap-cursor operand
// loads
// The two launches of a column split as one (gemm_pair_kernel): only for a
// one-split unit-geometry plan of 256 x 256 then 256 x 128 tiles with as many
// tiles in both parts; otherwise kPairNotApplicable and the caller launches
// the two parts.  MEMSAVE_GEMM_PAIR=off forces the two launches (testing knob).
constexpr int kPairNotApplicable = -2;
template <int MODE>
int go_pair(const Tile &t1, const Args &a1, const Tile &t2, const Args &a2, hipStream_t st) {
    const char *e = getenv("MEMSAVE_GEMM_PAIR");
    if (e && strcmp(e, "off") == 0) return kPairNotApplicable;
    if (!(t1.bm == 256 && t1.bn == 256 && t1.kg == 1 && t2.bm == 256 && t2.bn == 128 && t2.kg == 1 &&
          t2.stages == 3 && t1.stages == 2))
        return kPairNotApplicable;
    if (a1.splits > 1 || a2.splits > 1) return kPairNotApplicable;
    const int nb = a1.ntm * a1.ntn;
    if (nb != a2.ntm * a2.ntn || nb <= 0) return kPairNotApplicable;
    const unsigned pk = MODE == kFwd ? kProfFwd : kProfDgrad;
    void *eb = nullptr, *ee = nullptr;
    const bool timed = prof_pair(pk, &eb, &ee);
    hipExtLaunchKernelGGL(gemm_pair_kernel<MODE>, dim3(nb), dim3(512), 0, st, (hipEvent_t)eb, (hipEvent_t)ee, 0,
                          a1, a2);
    const int err = (int)hipGetLastError();
    if (timed) prof_pair_done(pk, eb, ee, err == 0);
    return err;
}

template <int MODE>
int go_mode(const Tile &t, const Args &a, dim3 grid, bool unit, hipStream_t st, bool ts = false) {
    if (unit) return go_tile<MODE, true>(t, a, grid, st);
    if constexpr (MODE == kFwd || MODE == kDgrad || MODE == kWgrad) {
        if (ts) return go_tile<MODE, false, true>(t, a, grid, st);
    }
    return go_tile<MODE, false>(t, a, grid, st);
}

bool al16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool unit_geom(const ConvGeom &g) {
    return g.R == 1 && g.S == 1 && g.sh == 1 && g.sw == 1 && g.ph == 0 && g.pw == 0 && g.P == g.H && g.Q == g.W;
}

// Byte size of an operand for its buffer descriptor; callers have checked
// operand_fits, so the size and every row base fit 32 bits.
uint32_t bytes_of(long elems) { return (uint32_t)(elems * 2); }

int pad8(int c) { return (c + 7) / 8 * 8; }
size_t al256(size_t n) { return (n + 255) / 256 * 256; }

int pad_channels(const void *src, int64_t rows, int C, void *dst, hipStream_t st) {
    const int C8 = pad8(C);
    const int64_t total = rows * (C8 / 8);
    if (total == 0) return 0;
    const int blocks = (int)std::min<int64_t>((total + 255) / 256, 8192);
    hipLaunchKernelGGL(pad_channels_kernel, dim3(blocks), dim3(256), 0, st, (const bf16 *)src, rows, C, C8, (bf16 *)dst);
    return (int)hipGetLastError();
}

int crop_channels(const void *src, int64_t rows, int C, void *dst, hipStream_t st) {
    const int64_t total = rows * C;
    if (total == 0) return 0;
    const int blocks = (int)std::min<int64_t>((total + 255) / 256, 8192);
    hipLaunchKernelGGL(crop_channels_kernel, dim3(blocks), dim3(256), 0, st, (const bf16 *)src, rows, pad8(C), C,
                       (bf16 *)dst);
    return (int)hipGetLastError();
}

// Pair packing applies to inputs of at most 4 channels with a stride-2
// width whose packed output width equals the original (true unless the
// padded width is odd and S even).
int pair_width(const ConvGeom &g) { return (g.W + 2 * g.pw + 1) / 2; }
bool pair_applies(const ConvGeom &g) {
    return g.C <= 4 && g.sw == 2 && pair_width(g) - (g.S + 1) / 2 + 1 == g.Q;
}
ConvGeom paired(const ConvGeom &g) {
    ConvGeom q = g;
    q.C = 8;
    q.W = pair_width(g);
    q.S = (g.S + 1) / 2;
    q.sw = 1;
    q.pw = 0;
    return q;
}

int launch_grid(int64_t work) { return (int)std::max<int64_t>(1, std::min<int64_t>((work + 255) / 256, 8192)); }

int pack_pairs(const ConvGeom &g, const void *x, void *xq, hipStream_t st) {
    const int64_t rows = (int64_t)g.N * g.H, work = rows * pair_width(g);
    if (work == 0) return 0;
    hipLaunchKernelGGL(pack_pairs_kernel, dim3(launch_grid(work)), dim3(256), 0, st, (const bf16 *)x, rows, g.W, g.C,
                       pair_width(g), g.pw, (bf16 *)xq);
    return (int)hipGetLastError();
}

int pack_pair_filter(const ConvGeom &g, const void *w, void *wq, hipStream_t st) {
    const int64_t KR = (int64_t)g.K * g.R, work = KR * ((g.S + 1) / 2);
    if (work == 0) return 0;
    hipLaunchKernelGGL(pack_pair_filter_kernel, dim3(launch_grid(work)), dim3(256), 0, st, (const bf16 *)w, KR, g.S,
                       g.C, (g.S + 1) / 2, (bf16 *)wq);
    return (int)hipGetLastError();
}

int unpack_pairs(const ConvGeom &g, const void *dxq, void *dx, hipStream_t st) {
    const int64_t rows = (int64_t)g.N * g.H, work = rows * g.W * g.C;
    if (work == 0) return 0;
    hipLaunchKernelGGL(unpack_pairs_kernel, dim3(launch_grid(work)), dim3(256), 0, st, (const bf16 *)dxq, rows, g.W,
                       g.C, pair_width(g), g.pw, (bf16 *)dx);
    return (int)hipGetLastError();
}

int unpack_pair_filter(const ConvGeom &g, const void *dwq, void *dw, hipStream_t st) {
    const int64_t KR = (int64_t)g.K * g.R, work = KR * g.S * g.C;
    if (work == 0) return 0;
    hipLaunchKernelGGL(unpack_pair_filter_kernel, dim3(launch_grid(work)), dim3(256), 0, st, (const bf16 *)dwq, KR,
                       g.S, g.C, (g.S + 1) / 2, (bf16 *)dw);
    return (int)hipGetLastError();
}

// 2 x 2 block packing (input gradient only): applies to inputs of at most 4
// channels with stride 2 in both dimensions whose packed output extents
// equal the original ones.
int block_height(const ConvGeom &g) { return (g.H + 2 * g.ph + 1) / 2; }
bool block_applies(const ConvGeom &g) {
    return g.C <= 4 && g.sh == 2 && g.sw == 2 && block_height(g) - (g.R + 1) / 2 + 1 == g.P &&
           pair_width(g) - (g.S + 1) / 2 + 1 == g.Q;
}
ConvGeom blocked(const ConvGeom &g) {
    ConvGeom q = g;
    q.C = 16;
    q.H = block_height(g);
    q.W = pair_width(g);
    q.R = (g.R + 1) / 2;
    q.S = (g.S + 1) / 2;
    q.sh = q.sw = 1;
    q.ph = q.pw = 0;
    return q;
}
size_t block_x_bytes(const ConvGeom &g) { return al256((size_t)g.N * block_height(g) * pair_width(g) * 16 * 2); }
size_t block_w_bytes(const ConvGeom &g) { return al256((size_t)g.K * ((g.R + 1) / 2) * ((g.S + 1) / 2) * 16 * 2); }

int pack_block_filter(const ConvGeom &g, const void *w, void *wq, hipStream_t st) {
    const int64_t work = (int64_t)g.K * ((g.R + 1) / 2) * ((g.S + 1) / 2);
    if (work == 0) return 0;
    hipLaunchKernelGGL(pack_block_filter_kernel, dim3(launch_grid(work)), dim3(256), 0, st, (const bf16 *)w, g.K, g.R,
                       g.S, g.C, (g.R + 1) / 2, (g.S + 1) / 2, (bf16 *)wq);
    return (int)hipGetLastError();
}

int pack_blocks(const ConvGeom &g, const void *x, void *xq, hipStream_t st) {
    const int64_t work = (int64_t)g.N * block_height(g) * pair_width(g);
    if (work == 0) return 0;
    if (work > INT32_MAX || (int64_t)g.N * g.H * g.W * g.C * 2 >= (int64_t)kOOB) return (int)hipErrorInvalidValue;
    // rows of whole 16-byte vectors that fit the LDS rows, x 16-byte aligned:
    // one workgroup per block row, coalesced loads
    if ((g.W * g.C) % 8 == 0 && g.W * g.C <= kUnpackRowMax && al16(x)) {
        hipLaunchKernelGGL(pack_blocks_row_kernel, dim3((unsigned)((int64_t)g.N * block_height(g))), dim3(128), 0, st,
                           (const bf16 *)x, g.H, g.W, g.C, block_height(g), pair_width(g), g.ph, g.pw, (bf16 *)xq);
        return (int)hipGetLastError();
    }
    hipLaunchKernelGGL(pack_blocks_kernel, dim3(launch_grid(work)), dim3(256), 0, st, (const bf16 *)x, (uint32_t)g.N, g.H,
                       g.W, g.C, block_height(g), pair_width(g), g.ph, g.pw, (bf16 *)xq);
    return (int)hipGetLastError();
}

int unpack_blocks(const ConvGeom &g, const void *dxq, void *dx, hipStream_t st) {
    const int64_t NH = (int64_t)g.N * g.H, work = NH * pair_width(g);
    if (work == 0) return 0;
    if (work > INT32_MAX) return (int)hipErrorInvalidValue;
    // rows of whole 16-byte vectors that fit the LDS row, dx 16-byte aligned:
    // one workgroup per row, coalesced stores
    if ((g.W * g.C) % 8 == 0 && g.W * g.C <= kUnpackRowMax && al16(dx) && NH <= INT32_MAX) {
        hipLaunchKernelGGL(unpack_blocks_row_kernel, dim3((unsigned)NH), dim3(128), 0, st, (const bf16 *)dxq, g.H, g.W,
                           g.C, block_height(g), pair_width(g), g.ph, g.pw, (bf16 *)dx);
        return (int)hipGetLastError();
    }
    hipLaunchKernelGGL(unpack_blocks_kernel, dim3(launch_grid(work)), dim3(256), 0, st, (const bf16 *)dxq,
                       (uint32_t)NH, g.H, g.W, g.C, block_height(g), pair_width(g), g.ph, g.pw, (bf16 *)dx);
    return (int)hipGetLastError();
}

size_t pair_x_bytes(const ConvGeom &g) { return al256((size_t)g.N * g.H * pair_width(g) * 8 * 2); }
size_t pair_w_bytes(const ConvGeom &g) { return al256((size_t)g.K * g.R * ((g.S + 1) / 2) * 8 * 2); }

// The geometry with C padded to a multiple of 8.
ConvGeom padded(const ConvGeom &g) {
    ConvGeom g8 = g;
    g8.C = pad8(g.C);
    return g8;
}

struct WgradPlan {
    Tile t;
    int splits, k_split;
};

// Weight gradient of a convolution with taps (im2col-gathered x): the tile
// and split count that minimise (waves of blocks) x (time per wave), splitting
// the reduction until the CUs are full.  Measured faster than plan_gemm's
// choice on the 3x3 conv sweep (71 against 81 us), whose constants come from
// unit-stride contractions.
// Without the reduction's price the weight gradients took the most splits the
// CUs allowed (the 4x4 stride-2 decoder layer 128 -> 256 channels: 256 x 256
// tiles in 32 splits, 64 us; 128 x 128 in 8 splits, 40 us).
constexpr double kWgradRedUnits = 6.0;
// Tiles of the convolution weight gradient (pixel-cursor loads): 256 x 128
// and the 8-wave 128 x 128 tiles.  Forced-tile runs on the ResNet-18-shaped
// layers, the conv sweep and the decoder had one of them fastest on every
// shape; 128 x 64 and the 4-wave 128 x 128 were up to 25% slower, and the
// 256 x 256 tile keeps the generic loads.
constexpr bool kAutoWg[kNumTiles] = {false, true, false, true, false, true, false, false, false, false, false};

Tile pick_conv_wgrad(long M, long N, long K, int splits_allowed, int *splits_out) {
    const int z = 1;
    double best = 1e300;
    Tile bt = kTiles[0];
    int bs = 1;
    int forced = forced_tile();
    // no k-group or narrow weight gradient: plan as usual
    if (forced >= 0 && (kTiles[forced].kg > 1 || kc_only(kTiles[forced]))) forced = -1;
    for (int ti = 0; ti < kNumTiles; ++ti) {
        if (forced >= 0 ? ti != forced : !kAutoWg[ti]) continue;
        const Tile &t = kTiles[ti];
        if (t.kg > 1 || kc_only(t)) continue;   // none of these is built for the weight gradient
        const long tiles = ((M + t.bm - 1) / t.bm) * ((N + t.bn - 1) / t.bn) * z;
        const long conc = (long)kCUs * t.per_cu;
        // every split count up to the CUs' fill (ceil(fill / tiles) can spill
        // into a second wave where floor stays in one)
        const int max_sp = (int)std::max<long>(1, std::min<long>(splits_allowed, (2 * conc + tiles - 1) / tiles));
        for (int splits = 1; splits <= max_sp; ++splits) {
            const long blocks = tiles * splits;
            const long waves = (blocks + conc - 1) / conc;
            // blocks that actually share a CU in the fullest wave
            const long resident = std::min<long>(t.per_cu, (blocks + kCUs - 1) / kCUs);
            const double kper = (double)K / splits;
            const double eff = resident > 1 ? t.eff : t.eff1;
            // the split reduction's pass: every split writes and the reduction
            // reads M x N fp32 partials, priced at kWgradRedUnits per element and
            // split (8 bytes at about 3 TB/s, in the MFMA units of the first term)
            const double red = splits > 1 ? kWgradRedUnits * (double)M * N * splits : 0.0;
            const double cost = (double)waves * resident * t.bm * t.bn * (kper + 64.0) / eff + red;
            if (cost < best * 0.999) {
                best = cost;
                bt = t;
                bs = splits;
            }
        }
    }
    if (splits_out) *splits_out = bs;
    return bt;
}

WgradPlan wgrad_plan(const ConvGeom &g) {
    const long M = g.K, N = (long)g.R * g.S * g.C, K = (long)g.N * g.P * g.Q;
    if (unit_geom(g)) {
        // (the weight gradient has no k-group tile)
        const GemmPlan p = plan_gemm(M, N, K, 1, 16, true, kKgNever);
        return {p.t, p.splits, p.k_split};
    }
    int splits = 1;
    const int max_splits = (int)std::max<long>(1, K / (8 * BK));   // at least 8 BK steps per split
    Tile t = pick_conv_wgrad(M, N, K, max_splits, &splits);
    const int fs = forced_splits();
    if (fs) splits = fs;
    int k_split = (int)((K + splits - 1) / splits);
    k_split = std::max(BK, (k_split + BK - 1) / BK * BK);
    // forced: keep the count even if some splits are empty (their partials are zeros)
    if (!fs) splits = K > 0 ? (int)((K + k_split - 1) / k_split) : 1;
    return {t, splits, k_split};
}

}  // namespace

// Each returns -1 when the fast path does not apply, else a hipError_t.

// Sum `splits` partial arrays of n floats (pstride apart) to bf16 `out`,
// adding bias[i % ncol] when bias is given.
int reduce_partials(const float *part, int splits, int64_t n, int64_t pstride, bf16 *out, const bf16 *bias, int ncol,
                    hipStream_t st) {
    const int blocks = (int)std::max<int64_t>(1, std::min<int64_t>((n / 4 + 255) / 256, 4096));
    hipLaunchKernelGGL(reduce_kernel, dim3(blocks), dim3(256), 0, st, part, splits, n, pstride, out,
                       (const float *)nullptr, 0, (bf16 *)nullptr, bias, ncol);
    return (int)hipGetLastError();
}

// ---------------------------------------------------------------- halo convolution (host)
// MEMSAVE_CONV_HALO=off turns the halo kernel off (testing knob: the tests run
// both paths).
bool halo_enabled() {
    const char *e = getenv("MEMSAVE_CONV_HALO");
    return !(e && strcmp(e, "off") == 0);
}

// Output tile of the halo kernel for an output of P x Q pixels with R x S
// taps: the width split into the fewest column tiles of at most 32, then as
// many rows as fit both 256 pixels and a halo of at most halo_max_px pixels
// (a tile always computes 256 rows of MFMA tiles, so the largest tile is the
// cheapest per pixel).  False when no tile fits.
bool halo_tile(int Q, int R, int S, int *TH, int *TW, int ch = 64, bool oph = false) {
    if (Q <= 0) return false;
    const int ntw = (Q + 31) / 32;
    const int tw = (Q + ntw - 1) / ntw;
    const int maxpx = oph ? halo_max_px_oph() : ch == 64 ? halo_max_px<64>() : halo_max_px<16>();
    const int th = std::min(256 / tw, maxpx / (tw + S - 1) - (R - 1));
    if (th < 1) return false;
    *TH = th;
    *TW = tw;
    return true;
}

// The halo kernel's instantiations: up to 64 output channels with up to 9
// taps, or up to 32 with up to 16.
bool halo_shape_ok(int NO, int taps) {
    return NO % 8 == 0 && NO > 0 && ((NO <= 32 && taps <= 16) || (NO <= 64 && taps <= 9));
}

// Output phases of a stride-2 input gradient along one dimension (R taps,
// padding ph): phase a takes taps r = r0 + 2u (r0 = (a + ph) mod 2) reading
// dy at i + e_a - u (e_a = (a + ph - r0) / 2).  *lo = the least dy offset
// over both phases (the halo origin), *span = the halo taps (offsets lo ..
// max e_a).  False when a phase has no tap.
bool oph_span(int R, int ph, int *lo, int *span) {
    int lo_ = 1 << 20, hi = -(1 << 20);
    for (int a = 0; a < 2; ++a) {
        const int r0 = (a + ph) & 1, nu = (R - r0 + 1) / 2, e = (a + ph - r0) / 2;
        if (nu < 1) return false;
        lo_ = std::min(lo_, e - (nu - 1));
        hi = std::max(hi, e);
    }
    *lo = lo_;
    *span = hi - lo_ + 1;
    return true;
}

// The output phases' tile (on the phase image of the input gradient), or false.
bool oph_tile(int Wx, int R, int S, int pw, int ph, int *TH, int *TW, HaloArgs *a = nullptr) {
    int lor, hr, los, hs;
    if (!oph_span(R, ph, &lor, &hr) || !oph_span(S, pw, &los, &hs)) return false;
    if (!halo_tile((Wx + 1) / 2, hr, hs, TH, TW, 64, true)) return false;
    if (a) {
        a->hr = hr; a->hs = hs; a->lor = lor; a->los = los;
    }
    return true;
}

// in[N][H][W][ch] -> out[N][P][Q][NO] (see halo_conv_kernel); ch = 64, or
// 16 (33 to 64 outputs over exactly 16 taps, the stem's 2 x 2 blocks);
// stride 1, or 2 (64 channels, up to 64 outputs and 9 taps, not flipped:
// the four stride phases, each with at most ceil(R/2) x ceil(S/2) taps).
// oph: the input gradient of a stride-2 convolution (in = dy of H x W,
// out = dx of P x Q, ph / pw the convolution's padding, filt = Wt[NO][R][S][64]
// not flipped) as its four output phases.
int run_halo(const bf16 *in, int N, int H, int W, const bf16 *filt, const bf16 *bias, int NO, int R, int S, int ph,
             int pw, bool flip, bf16 *out, int P, int Q, hipStream_t st, int ch = 64, int stride = 1,
             bool oph = false) {
    HaloArgs a{};
    a.in = in; a.filt = filt; a.bias = bias; a.out = out;
    a.H = H; a.W = W; a.P = P; a.Q = Q; a.R = R; a.S = S; a.ph = ph; a.pw = pw;
    a.NO = NO; a.flip = flip ? 1 : 0;
    if (ch != 64 && !(ch == 16 && NO > 32 && NO <= 64 && R * S == 16)) return (int)hipErrorInvalidValue;
    if (stride != 1 && !(stride == 2 && ch == 64 && !flip && NO <= 64 && R * S <= 9)) return (int)hipErrorInvalidValue;
    if (oph && !(stride == 1 && ch == 64 && !flip && NO <= 64 && R * S <= 9)) return (int)hipErrorInvalidValue;
    if (oph ? !oph_tile(Q, R, S, pw, ph, &a.TH, &a.TW, &a)
            : !halo_tile(Q, (R + stride - 1) / stride, (S + stride - 1) / stride, &a.TH, &a.TW, ch))
        return (int)hipErrorInvalidValue;
    // output tiles over the output (OPH: over its phase image, ceil(P/2) x ceil(Q/2))
    const int tiles_h = ((oph ? (P + 1) / 2 : P) + a.TH - 1) / a.TH;
    a.tiles_w = ((oph ? (Q + 1) / 2 : Q) + a.TW - 1) / a.TW;
    a.tiles_img = tiles_h * a.tiles_w;
    const long tiles = (long)N * a.tiles_img;
    if (tiles == 0) return 0;
    if (tiles > INT32_MAX) return (int)hipErrorInvalidValue;
    a.tiles = (int)tiles;
    a.in_bytes = bytes_of((long)N * H * W * ch);
    a.filt_bytes = bytes_of((long)NO * R * S * ch);
    if (!operand_fits((long)N * P * Q * NO)) return (int)hipErrorInvalidValue;
    a.out_bytes = bytes_of((long)N * P * Q * NO);
    const dim3 grid((unsigned)std::min<long>(tiles, kCUs));
    const unsigned pk = flip || oph ? kProfDgrad : kProfFwd;   // the input-gradient contractions
    void *eb = nullptr, *ee = nullptr;
    const bool timed = prof_pair(pk, &eb, &ee);
    if (oph)
        hipExtLaunchKernelGGL((halo_conv_kernel<64, 9, 1, false, 64, 1, true>), grid, dim3(256), 0, st,
                              (hipEvent_t)eb, (hipEvent_t)ee, 0, a);
    else if (stride == 2)
        hipExtLaunchKernelGGL((halo_conv_kernel<64, 9, 1, false, 64, 2>), grid, dim3(256), 0, st, (hipEvent_t)eb,
                              (hipEvent_t)ee, 0, a);
    else if (ch == 16)
        hipExtLaunchKernelGGL((halo_conv_kernel<64, 16, 1, true, 16>), grid, dim3(256), 0, st, (hipEvent_t)eb,
                              (hipEvent_t)ee, 0, a);
    else if (NO <= 32 && R * S == 16)   // 4 x 4: the unrolled schedule
        hipExtLaunchKernelGGL((halo_conv_kernel<32, 16, 2, true>), grid, dim3(512), 0, st, (hipEvent_t)eb, (hipEvent_t)ee, 0, a);
    else if (NO <= 32)
        hipExtLaunchKernelGGL((halo_conv_kernel<32, 16, 2>), grid, dim3(512), 0, st, (hipEvent_t)eb, (hipEvent_t)ee, 0, a);
    else if (R * S == 9)   // 3 x 3: the unrolled schedule
        hipExtLaunchKernelGGL((halo_conv_kernel<64, 9, 1, true>), grid, dim3(256), 0, st, (hipEvent_t)eb, (hipEvent_t)ee, 0, a);
    else
        hipExtLaunchKernelGGL((halo_conv_kernel<64, 9, 1>), grid, dim3(256), 0, st, (hipEvent_t)eb, (hipEvent_t)ee, 0, a);
    const int err = (int)hipGetLastError();
    if (timed) prof_pair_done(pk, eb, ee, err == 0);
    return err;
}

// Forward of a layer with at most 4 input channels and stride 2 (the stem)
// through 2 x 2 pixel blocks: a stride-1 convolution of 16-channel blocks
// with 4 x 4 taps, 33 to 64 outputs (a multiple of 8).
bool halo_block_fwd_applies(const ConvGeom &g) {
    if (!halo_enabled() || !block_applies(g) || (g.R + 1) / 2 != 4 || (g.S + 1) / 2 != 4) return false;
    if (g.K % 8 != 0 || g.K <= 32 || g.K > 64) return false;
    const ConvGeom q = blocked(g);
    int th, tw;
    return operand_fits((long)g.N * g.P * g.Q * g.K) && operand_fits((long)q.N * q.H * q.W * 16) &&
           halo_tile(g.Q, 4, 4, &th, &tw, 16);
}

// Forward: 64 input channels, the filter within the kernel's
// instantiations, more than one tap; stride 1, or 2 with up to 64 outputs
// and 9 taps (its stride phases).
bool halo_fwd_applies(const ConvGeom &g) {
    const bool s1 = g.sh == 1 && g.sw == 1, s2 = g.sh == 2 && g.sw == 2 && g.K <= 64 && g.R * g.S <= 9;
    const int st = s2 ? 2 : 1;
    return halo_enabled() && g.C == 64 && (s1 || s2) && g.R * g.S > 1 && halo_shape_ok(g.K, g.R * g.S) &&
           g.P > 0 && g.Q > 0 && operand_fits((long)g.N * g.P * g.Q * g.K) &&
           [&] { int th, tw; return halo_tile(g.Q, (g.R + st - 1) / st, (g.S + st - 1) / st, &th, &tw); }();
}

// Input gradient: the correlation of dy (64 channels) with the flipped,
// transposed filter and padding R - 1 - ph (stride 1), or (stride 2, up to
// 64 input channels and 9 taps) its four output phases.
bool halo_dgrad_s2(const ConvGeom &g) {
    int th, tw;
    return g.sh == 2 && g.sw == 2 && g.C <= 64 && g.R * g.S <= 9 && oph_tile(g.W, g.R, g.S, g.pw, g.ph, &th, &tw);
}
bool halo_dgrad_applies(const ConvGeom &g) {
    if (!halo_enabled() || g.K != 64 || g.R * g.S <= 1 || !halo_shape_ok(g.C, g.R * g.S) || g.H <= 0 || g.W <= 0 ||
        !operand_fits((long)g.N * g.H * g.W * g.C))
        return false;
    if (g.sh == 1 && g.sw == 1)
        return g.ph <= g.R - 1 && g.pw <= g.S - 1 && [&] { int th, tw; return halo_tile(g.W, g.R, g.S, &th, &tw); }();
    return halo_dgrad_s2(g);
}

// The convolution forward and input gradient run on the tap-step operand
// loads when each BK-deep step lies in one tap.
bool ts_fwd(const ConvGeom &g) { return !unit_geom(g) && g.C % BK == 0 && g.R * g.S <= 32; }
bool ts_dgrad(const ConvGeom &g) {
    return !unit_geom(g) && g.K % BK == 0 && ((g.R + g.sh - 1) / g.sh) * ((g.S + g.sw - 1) / g.sw) <= 32;
}

GemmPlan fwd_plan(const ConvGeom &g) {
    return plan_gemm((long)g.N * g.P * g.Q, g.K, (long)g.R * g.S * g.C, 1, 16, true, kKgAuto,
                     ts_fwd(g) ? kAutoTs : unit_geom(g) ? kAutoUnitKc : kAutoKc);
}

size_t fwd_split_bytes(const ConvGeom &g) {
    const GemmPlan p = fwd_plan(g);
    if (p.splits <= 1) return 0;
    return al256((size_t)p.splits * part_stride((int64_t)g.N * g.P * g.Q * g.K) * sizeof(float));
}

// Forward with C % 8 != 0: padded copies of x and W, then the workspace of
// the padded contraction (split-K partials).
size_t fwd_workspace(const ConvGeom &g) {
    if (g.C % 8 == 0) return fwd_split_bytes(g);
    if (halo_block_fwd_applies(g)) return block_x_bytes(g) + block_w_bytes(g);
    if (pair_applies(g)) return pair_x_bytes(g) + pair_w_bytes(g) + fwd_split_bytes(paired(g));
    const int C8 = pad8(g.C);
    return al256((size_t)g.N * g.H * g.W * C8 * 2) + al256((size_t)g.K * g.R * g.S * C8 * 2) +
           fwd_split_bytes(padded(g));
}

int conv_fwd(const ConvGeom &g, const void *x, const void *w, const void *bias, void *y, void *ws, hipStream_t st) {
    if (g.C % 8 != 0 && halo_block_fwd_applies(g)) {
        // the stem: 2 x 2 pixel blocks, a stride-1 4 x 4 convolution of 16 channels
        if (!ws || !al16(ws) || !al16(y)) return -1;
        char *xq = static_cast<char *>(ws);
        char *wq = xq + block_x_bytes(g);
        int err = pack_blocks(g, x, xq, st);
        if (!err) err = pack_block_filter(g, w, wq, st);
        if (err) return err;
        const ConvGeom q = blocked(g);
        return run_halo((const bf16 *)xq, q.N, q.H, q.W, (const bf16 *)wq, (const bf16 *)bias, g.K, 4, 4, 0, 0, false,
                        (bf16 *)y, g.P, g.Q, st, 16);
    }
    if (g.C % 8 != 0 && pair_applies(g)) {
        if (!ws || !al16(ws) || !al16(y)) return -1;
        char *xq = static_cast<char *>(ws);
        char *wq = xq + pair_x_bytes(g);
        char *ws2 = wq + pair_w_bytes(g);
        int err = pack_pairs(g, x, xq, st);
        if (!err) err = pack_pair_filter(g, w, wq, st);
        if (err) return err;
        return conv_fwd(paired(g), xq, wq, bias, y, ws2, st);
    }
    if (g.C % 8 != 0) {
        if (!ws || !al16(ws) || !al16(y)) return -1;
        const ConvGeom g8 = padded(g);
        char *xp = static_cast<char *>(ws);
        char *wp = xp + al256((size_t)g.N * g.H * g.W * g8.C * 2);
        char *ws2 = wp + al256((size_t)g.K * g.R * g.S * g8.C * 2);
        int err = pad_channels(x, (int64_t)g.N * g.H * g.W, g.C, xp, st);
        if (!err) err = pad_channels(w, (int64_t)g.K * g.R * g.S, g.C, wp, st);
        if (err) return err;
        return conv_fwd(g8, xp, wp, bias, y, ws2, st);
    }
    if (!al16(x) || !al16(w) || !al16(y)) return -1;
    if (!operand_fits((long)g.N * g.H * g.W * g.C) || !operand_fits((long)g.K * g.R * g.S * g.C)) return -1;
    if (halo_fwd_applies(g))
        return run_halo((const bf16 *)x, g.N, g.H, g.W, (const bf16 *)w, (const bf16 *)bias, g.K, g.R, g.S, g.ph, g.pw,
                        false, (bf16 *)y, g.P, g.Q, st, 64, g.sh);
    Args a{};
    a.a = (const bf16 *)x; a.b = (const bf16 *)w; a.c = (bf16 *)y; a.g = g;
    a.M = g.N * g.P * g.Q; a.N = g.K; a.K = g.R * g.S * g.C;
    if (a.M == 0 || a.N == 0) return 0;
    const GemmPlan p = fwd_plan(g);
    if (p.splits > 1 && (!ws || !al16(ws))) return -1;
    a.ntm = (a.M + p.t.bm - 1) / p.t.bm; a.ntn = (a.N + p.t.bn - 1) / p.t.bn;
    a.splits = p.splits; a.k_split = p.k_split;
    a.a_bytes = bytes_of((long)g.N * g.H * g.W * g.C);
    a.b_bytes = bytes_of((long)g.K * a.K);
    const int64_t n = (int64_t)a.M * a.N;
    if (p.splits > 1) {
        a.part = static_cast<float *>(ws);
        a.part_stride = part_stride(n);
        a.c = nullptr;
    } else {
        a.bias = (const bf16 *)bias;
    }
    const ColSplit cs = unit_geom(g) ? col_split(p, a.M, a.N, a.K, kAutoKc) : ColSplit{};
    if (cs.n1 > 0) {
        // filter rows and output columns [0, n1), then [n1, K)
        Args a2 = a;
        a.N = cs.n1;
        a.ldc = g.K;
        a.ntn = (a.N + p.t.bn - 1) / p.t.bn;
        a2.b += (size_t)cs.n1 * a2.K;
        a2.c += cs.n1;
        if (a2.bias) a2.bias += cs.n1;
        a2.N = g.K - cs.n1;
        a2.ldc = g.K;
        a2.b_bytes = bytes_of((long)a2.N * a2.K);
        a2.ntm = (a2.M + cs.p2.t.bm - 1) / cs.p2.t.bm;
        a2.ntn = (a2.N + cs.p2.t.bn - 1) / cs.p2.t.bn;
        a2.k_split = cs.p2.k_split;
        const int pr = go_pair<kFwd>(p.t, a, cs.p2.t, a2, st);
        if (pr != kPairNotApplicable) return pr;
        const int err = go_mode<kFwd>(p.t, a, dim3(a.ntm * a.ntn), true, st);
        if (err) return err;
        return go_mode<kFwd>(cs.p2.t, a2, dim3(a2.ntm * a2.ntn), true, st);
    }
    int err = go_mode<kFwd>(p.t, a, dim3(a.ntm * a.ntn, 1, p.splits), unit_geom(g), st, ts_fwd(g));
    if (err || p.splits <= 1) return err;
    return reduce_partials(a.part, p.splits, n, a.part_stride, (bf16 *)y, (const bf16 *)bias, a.N, st);
}

// Input gradient either straight from W (filter read in place through
// transposing LDS reads; no copy, no extra kernel, no split) or through a
// transposed copy Wt[C][R][S][K] (both operands K-contiguous).  An 8-wave
// tile hides the transposing reads (within 2% of the copy's contraction), so
// W is read in place unless the plan wants a 4-wave tile (which does not) or
// a split reduction (which only the copy's contraction has).  The strided
// variant through the copy has no 256 x 256 tile.
// MEMSAVE_DGRAD=transposed|direct overrides the choice (testing knob).
struct DgradChoice {
    bool direct;
    GemmPlan p;
};

DgradChoice dgrad_choice(const ConvGeom &g) {
    // GEMM bounds over the stride phases: ceil(H/sh) x ceil(W/sw) rows per
    // image, ceil(R/sh) x ceil(S/sw) taps
    const long Hb = (g.H + g.sh - 1) / g.sh, Wb = (g.W + g.sw - 1) / g.sw;
    const long Kb = (long)((g.R + g.sh - 1) / g.sh) * ((g.S + g.sw - 1) / g.sw) * g.K;
    const long M = (long)g.N * Hb * Wb;
    const int z = g.sh * g.sw;
    const bool unit = unit_geom(g);
    const int kg = unit ? kKgAuto : kKgForced;
    const bool *set = unit ? kAutoKc : ts_dgrad(g) ? kAutoTs : kAutoConv;
    const char *e = getenv("MEMSAVE_DGRAD");
    const int forced = forced_tile();
    // the narrow and 192-wide tiles read W through the transposed copy only
    const bool kc_forced = forced >= 0 && kc_only(kTiles[forced]);
    if (e && *e && !kc_forced) {
        const bool direct = e[0] == 'd';
        return {direct, plan_gemm(M, g.C, Kb, z, direct ? 1 : 16, direct || unit, kg, direct ? kAuto : set)};
    }
    const GemmPlan pt = plan_gemm(M, g.C, Kb, z, 16, unit, kg, set);
    if (!unit) return {false, pt};
    if (narrow_tile(pt.t) || kc_forced) return {false, pt};
    const GemmPlan pd = plan_gemm(M, g.C, Kb, z, 1, true, kg);
    const bool pd_ok = pd.t.wr * pd.t.wc * pd.t.kg == 8 && pt.splits == 1 && !kc_only(pd.t);
    if (kc_only(pt.t)) {
        // the 192-wide tile pays the transposed copy (read and write W once
        // plus a launch); the in-place variant pays nothing extra
        const double tr_us = 1.0 + 4.0 * (double)g.K * g.R * g.S * g.C / kBytesPerUs;
        if (pd_ok && est_us(pd.t, M, g.C, Kb, z, 1) <= est_us(pt.t, M, g.C, Kb, z, pt.splits) + tr_us) return {true, pd};
        return {false, pt};
    }
    if (pd_ok) return {true, pd};
    return {false, pt};
}

// The bias gradient rides on a unit-geometry input gradient that does not
// split its reduction: every block also adds its share of dy's columns
// (dy_column_sums), leaving one partial row per (row tile, summing wave).
bool colsum_rides(const ConvGeom &g, const GemmPlan &p) { return unit_geom(g) && p.splits == 1; }
int colsum_waves(const Tile &t) { return t.wr * t.wc; }   // k-groups: the second group's waves
int64_t colsum_rows(const ConvGeom &g, const Tile &t) {
    return (((int64_t)g.N * g.H * g.W + t.bm - 1) / t.bm) * colsum_waves(t);
}

// transposed filter (when used), then split-K partials indexed by dx pixel,
// then (with_db, when the column sums ride along) their partial rows
size_t dgrad_core_workspace(const ConvGeom &g, bool with_db) {
    if (halo_dgrad_applies(g)) return al256((size_t)g.K * g.R * g.S * g.C * sizeof(bf16));   // the transposed filter
    const DgradChoice dc = dgrad_choice(g);
    const GemmPlan &p = dc.p;
    size_t ws = dc.direct ? 0 : al256((size_t)g.K * g.R * g.S * g.C * sizeof(bf16));
    if (p.splits > 1) ws += al256((size_t)p.splits * part_stride((int64_t)g.N * g.H * g.W * g.C) * sizeof(float));
    if (with_db && colsum_rides(g, p)) ws += al256((size_t)colsum_rows(g, p.t) * g.K * sizeof(float));
    return ws;
}

size_t dgrad_workspace(const ConvGeom &g, bool with_db) {
    if (g.K % 8 != 0) return 0;
    if (g.C % 8 != 0) {
        // block or pair packing (without a bias) or channel padding, whichever is larger
        const size_t bq = block_applies(g) ? block_w_bytes(g) + block_x_bytes(g) + dgrad_core_workspace(blocked(g), false) : 0;
        const size_t pq = std::max(bq, pair_applies(g) ? pair_w_bytes(g) + pair_x_bytes(g) + dgrad_core_workspace(paired(g), false) : 0);
        // padded W, padded bias, padded dx, then the workspace of the padded
        // contraction
        const ConvGeom g8 = padded(g);
        return std::max(pq, al256((size_t)g.K * g.R * g.S * g8.C * 2) + al256((size_t)g8.C * 2) +
                                al256((size_t)g.N * g.H * g.W * g8.C * 2) + dgrad_core_workspace(g8, false));
    }
    return dgrad_core_workspace(g, with_db);
}

// dx = input gradient (+ bias[c] per channel when bias is non-null: the
// forward of a transposed convolution runs this contraction).  With db
// non-null the contraction may also produce db[k] = sum of dy's column k
// (the layer's bias gradient); *db_done says whether it did.
int conv_dgrad(const ConvGeom &g, const void *dy, const void *w, const void *bias, void *dx, void *ws,
               hipStream_t st, void *db, bool *db_done) {
    if (db_done) *db_done = false;
    if (g.K % 8 != 0) return -1;
    if (g.C % 8 != 0 && block_applies(g) && !bias) {
        if (!ws || !al16(ws)) return -1;
        char *wq = static_cast<char *>(ws);
        char *dxq = wq + block_w_bytes(g);
        char *ws2 = dxq + block_x_bytes(g);
        int err = pack_block_filter(g, w, wq, st);
        if (err) return err;
        err = conv_dgrad(blocked(g), dy, wq, nullptr, dxq, ws2, st, nullptr, nullptr);
        if (err) return err;   // -1: not applicable (the caller falls back), else a HIP error
        return unpack_blocks(g, dxq, dx, st);
    }
    if (g.C % 8 != 0 && pair_applies(g) && !bias) {
        if (!ws || !al16(ws)) return -1;
        char *wq = static_cast<char *>(ws);
        char *dxq = wq + pair_w_bytes(g);
        char *ws2 = dxq + pair_x_bytes(g);
        int err = pack_pair_filter(g, w, wq, st);
        if (err) return err;
        err = conv_dgrad(paired(g), dy, wq, nullptr, dxq, ws2, st, nullptr, nullptr);
        if (err) return err;   // -1: not applicable (the caller falls back), else a HIP error
        return unpack_pairs(g, dxq, dx, st);
    }
    if (g.C % 8 != 0) {
        if (!ws || !al16(ws)) return -1;
        const ConvGeom g8 = padded(g);
        char *wp = static_cast<char *>(ws);
        char *bp = wp + al256((size_t)g.K * g.R * g.S * g8.C * 2);
        char *dxp = bp + al256((size_t)g8.C * 2);
        char *ws2 = dxp + al256((size_t)g.N * g.H * g.W * g8.C * 2);
        int err = pad_channels(w, (int64_t)g.K * g.R * g.S, g.C, wp, st);
        if (!err && bias) err = pad_channels(bias, 1, g.C, bp, st);
        if (err) return err;
        err = conv_dgrad(g8, dy, wp, bias ? bp : nullptr, dxp, ws2, st, nullptr, nullptr);
        if (err) return err;   // -1: not applicable (the caller falls back), else a HIP error
        return crop_channels(dxp, (int64_t)g.N * g.H * g.W, g.C, dx, st);
    }
    if (!al16(dy) || !al16(w) || !al16(dx)) return -1;
    if (!operand_fits((long)g.N * g.P * g.Q * g.K) || !operand_fits((long)g.K * g.R * g.S * g.C)) return -1;
    if (halo_dgrad_applies(g)) {
        // the correlation of dy with the flipped, transposed filter Wt[c][r][s][k]
        if (!ws || !al16(ws)) return -1;
        bf16 *wt = reinterpret_cast<bf16 *>(ws);
        const int err = transpose_krsc(w, wt, g.K, g.R * g.S, g.C, st);
        if (err) return err;
        if (g.sh == 2)   // the four output phases
            return run_halo((const bf16 *)dy, g.N, g.P, g.Q, wt, (const bf16 *)bias, g.C, g.R, g.S, g.ph, g.pw, false,
                            (bf16 *)dx, g.H, g.W, st, 64, 1, true);
        return run_halo((const bf16 *)dy, g.N, g.P, g.Q, wt, (const bf16 *)bias, g.C, g.R, g.S, g.R - 1 - g.ph,
                        g.S - 1 - g.pw, true, (bf16 *)dx, g.H, g.W, st);
    }
    const DgradChoice dc = dgrad_choice(g);
    const bool direct = dc.direct;
    const GemmPlan &p = dc.p;
    if ((!direct || p.splits > 1) && (!ws || !al16(ws))) return -1;
    char *wsc = static_cast<char *>(ws);
    bf16 *wt = direct ? nullptr : reinterpret_cast<bf16 *>(wsc);
    float *part = nullptr;
    if (p.splits > 1) part = reinterpret_cast<float *>(wsc + (direct ? 0 : al256((size_t)g.K * g.R * g.S * g.C * sizeof(bf16))));
    Args a{};
    a.a = (const bf16 *)dy; a.b = direct ? (const bf16 *)w : wt; a.c = (bf16 *)dx; a.g = g;
    a.bias = (const bf16 *)bias;
    const int Hb = (g.H + g.sh - 1) / g.sh, Wb = (g.W + g.sw - 1) / g.sw;
    a.M = g.N * Hb * Wb; a.N = g.C;
    a.K = ((g.R + g.sh - 1) / g.sh) * ((g.S + g.sw - 1) / g.sw) * g.K;
    if (a.M == 0 || a.N == 0) return 0;
    if (!direct) {
        const int err = transpose_krsc(w, wt, g.K, g.R * g.S, g.C, st);
        if (err) return err;
    }
    a.ntm = (a.M + p.t.bm - 1) / p.t.bm; a.ntn = (a.N + p.t.bn - 1) / p.t.bn;
    a.splits = p.splits; a.k_split = p.k_split;
    a.a_bytes = bytes_of((long)g.N * g.P * g.Q * g.K);
    a.b_bytes = bytes_of((long)g.K * g.R * g.S * g.C);
    const int64_t n = (int64_t)g.N * g.H * g.W * g.C;
    if (p.splits > 1) {
        a.part = part;
        a.part_stride = part_stride(n);
        a.c = nullptr;
    }
    const bool cs = db && !bias && colsum_rides(g, p);
    if (cs) {
        a.cspart = reinterpret_cast<float *>(wsc + (direct ? 0 : al256((size_t)g.K * g.R * g.S * g.C * sizeof(bf16))));
        a.cs_cw = (g.K + a.ntn - 1) / a.ntn;
        a.cs_cw = (a.cs_cw + 7) / 8 * 8;
    }
    const ColSplit tsp = !cs && unit_geom(g) ? col_split(p, a.M, a.N, a.K, direct ? kAuto : kAutoKc) : ColSplit{};
    if (tsp.n1 > 0) {
        // dx columns [0, n1), then [n1, C): W in place is [K][C] (columns
        // along its rows), the transposed copy [C][K] (one row per column)
        Args a2 = a;
        a.N = tsp.n1;
        a.ldc = g.C;
        a.ntn = (a.N + p.t.bn - 1) / p.t.bn;
        a2.b += direct ? (size_t)tsp.n1 : (size_t)tsp.n1 * g.K;
        a2.c += tsp.n1;
        if (a2.bias) a2.bias += tsp.n1;
        a2.N = g.C - tsp.n1;
        a2.ldc = g.C;
        a2.b_bytes = direct ? bytes_of((long)g.K * g.C - tsp.n1) : bytes_of((long)a2.N * g.K);
        a2.ntm = (a2.M + tsp.p2.t.bm - 1) / tsp.p2.t.bm;
        a2.ntn = (a2.N + tsp.p2.t.bn - 1) / tsp.p2.t.bn;
        a2.k_split = tsp.p2.k_split;
        const int pr = direct ? go_pair<kDgradN>(p.t, a, tsp.p2.t, a2, st) : go_pair<kDgrad>(p.t, a, tsp.p2.t, a2, st);
        if (pr != kPairNotApplicable) return pr;
        const int err = direct ? go_mode<kDgradN>(p.t, a, dim3(a.ntm * a.ntn), true, st)
                               : go_mode<kDgrad>(p.t, a, dim3(a.ntm * a.ntn), true, st);
        if (err) return err;
        return direct ? go_mode<kDgradN>(tsp.p2.t, a2, dim3(a2.ntm * a2.ntn), true, st)
                      : go_mode<kDgrad>(tsp.p2.t, a2, dim3(a2.ntm * a2.ntn), true, st);
    }
    const dim3 grid(a.ntm * a.ntn, 1, g.sh * g.sw * p.splits);
    int err = direct ? go_mode<kDgradN>(p.t, a, grid, unit_geom(g), st)
                     : go_mode<kDgrad>(p.t, a, grid, unit_geom(g), st, ts_dgrad(g));
    if (err) return err;
    if (cs) {
        err = launch_colsum_finalize(kBF16, a.cspart, (int)colsum_rows(g, p.t), g.K, db, st);
        if (!err && db_done) *db_done = true;
        return err;
    }
    if (p.splits <= 1) return err;
    return reduce_partials(part, p.splits, n, a.part_stride, (bf16 *)dx, (const bf16 *)bias, g.C, st);
}

bool wgrad_applies(const ConvGeom &g) { return g.K % 8 == 0; }

size_t wgrad_workspace(const ConvGeom &g, bool with_db) {
    if (g.C % 8 != 0 && pair_applies(g))
        return pair_x_bytes(g) + pair_w_bytes(g) + wgrad_workspace(paired(g), with_db);
    if (g.C % 8 != 0) {
        // padded x, padded dW, then the workspace of the padded contraction
        const ConvGeom g8 = padded(g);
        return al256((size_t)g.N * g.H * g.W * g8.C * 2) + al256((size_t)g.K * g.R * g.S * g8.C * 2) +
               wgrad_workspace(g8, with_db);
    }
    WgradPlan p = wgrad_plan(g);
    size_t ws = 0;
    if (p.splits > 1) ws += (size_t)p.splits * g.K * ((size_t)g.R * g.S * g.C) * sizeof(float);
    if (with_db) ws += (size_t)p.splits * g.K * sizeof(float);
    return ws;
}

int conv_wgrad(const ConvGeom &g, const void *dy, const void *x, void *dw, void *db, void *ws, hipStream_t st) {
    if (!wgrad_applies(g)) return -1;
    if (g.C % 8 != 0 && pair_applies(g)) {
        if (!ws || !al16(ws) || !al16(dy)) return -1;
        char *xq = static_cast<char *>(ws);
        char *dwq = xq + pair_x_bytes(g);
        char *ws2 = dwq + pair_w_bytes(g);
        int err = pack_pairs(g, x, xq, st);
        if (err) return err;
        err = conv_wgrad(paired(g), dy, xq, dwq, db, ws2, st);
        if (err) return err;   // -1: not applicable (the caller falls back), else a HIP error
        return unpack_pair_filter(g, dwq, dw, st);
    }
    if (g.C % 8 != 0) {
        if (!ws || !al16(ws) || !al16(dy)) return -1;
        const ConvGeom g8 = padded(g);
        char *xp = static_cast<char *>(ws);
        char *dwp = xp + al256((size_t)g.N * g.H * g.W * g8.C * 2);
        char *ws2 = dwp + al256((size_t)g.K * g.R * g.S * g8.C * 2);
        int err = pad_channels(x, (int64_t)g.N * g.H * g.W, g.C, xp, st);
        if (err) return err;
        err = conv_wgrad(g8, dy, xp, dwp, db, ws2, st);
        if (err) return err;   // -1: not applicable (the caller falls back), else a HIP error
        return crop_channels(dwp, (int64_t)g.K * g.R * g.S, g.C, dw, st);
    }
    if (!al16(dy) || !al16(x) || !al16(dw)) return -1;
    if (!operand_fits((long)g.N * g.P * g.Q * g.K) || !operand_fits((long)g.N * g.H * g.W * g.C)) return -1;
    WgradPlan p = wgrad_plan(g);
    Args a{};
    a.a = (const bf16 *)dy; a.b = (const bf16 *)x; a.g = g;
    a.M = g.K; a.N = g.R * g.S * g.C; a.K = g.N * g.P * g.Q;
    if (a.M == 0 || a.N == 0) return 0;
    a.ntm = (a.M + p.t.bm - 1) / p.t.bm; a.ntn = (a.N + p.t.bn - 1) / p.t.bn;
    a.splits = p.splits; a.k_split = p.k_split;
    float *wsf = static_cast<float *>(ws);
    size_t used = 0;
    if (p.splits > 1) {
        a.part = wsf;
        a.part_stride = (int64_t)a.M * a.N;
        used = (size_t)p.splits * a.M * a.N;
        a.c = nullptr;
    } else {
        a.c = (bf16 *)dw;
    }
    a.dbpart = db ? wsf + used : nullptr;
    a.a_bytes = bytes_of((long)g.N * g.P * g.Q * g.K);
    a.b_bytes = bytes_of((long)g.N * g.H * g.W * g.C);
    int err = go_mode<kWgrad>(p.t, a, dim3(a.ntm * a.ntn, 1, p.splits), unit_geom(g), st, true);
    if (err) return err;
    if (p.splits > 1 || db) {
        const int64_t n = p.splits > 1 ? (int64_t)a.M * a.N : 0;
        const int blocks = (int)std::max<int64_t>(1, std::min<int64_t>((n / 4 + 255) / 256, 2048));
        hipLaunchKernelGGL(reduce_kernel, dim3(blocks), dim3(256), 0, st, (const float *)a.part, p.splits, n, n,
                           (bf16 *)dw, (const float *)a.dbpart, db ? a.M : 0, (bf16 *)db, (const bf16 *)nullptr, 1);
        err = (int)hipGetLastError();
    }
    return err;
}

}  // namespace g2

int gemm_plan_info(int pass, const ConvGeom &g, int out[10]) {
    for (int i = 0; i < 10; ++i) out[i] = 0;
    if (g.C % 8 != 0 || g.K % 8 != 0 || pass < 0 || pass > 2) return -1;
    auto put = [&](const g2::Tile &t, int splits) {
        out[0] = t.bm;
        out[1] = t.bn;
        out[2] = t.wr * t.wc * t.kg;
        out[3] = t.stages;
        out[4] = t.kg;
        out[5] = splits;
    };
    auto put2 = [&](const g2::ColSplit &c) {
        out[7] = c.n1;
        if (c.n1 > 0) {
            out[8] = c.p2.t.bm;
            out[9] = c.p2.t.bn;
        }
    };
    const bool unit = g2::unit_geom(g);
    if (pass == 0) {
        const g2::GemmPlan p = g2::fwd_plan(g);
        put(p.t, p.splits);
        if (unit) put2(g2::col_split(p, (long)g.N * g.P * g.Q, g.K, (long)g.R * g.S * g.C, g2::kAutoKc));
    } else if (pass == 1) {
        const g2::DgradChoice d = g2::dgrad_choice(g);
        put(d.p.t, d.p.splits);
        out[6] = d.direct ? 1 : 0;
        if (unit) put2(g2::col_split(d.p, (long)g.N * g.H * g.W, g.C, g.K, d.direct ? g2::kAuto : g2::kAutoKc));
    } else {
        const g2::WgradPlan w = g2::wgrad_plan(g);
        put(w.t, w.splits);
    }
    return 0;
}

}  // namespace ms
