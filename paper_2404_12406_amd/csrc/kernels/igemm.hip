// Implicit-GEMM convolution kernels for gfx950 (MFMA), NHWC activations and
// KRSC filters.  One kernel template covers the three contractions of a
// layer that is linear in input and weight (Sec. 2.2.1 of the paper):
//
//   FWD    y[m][n]   = sum_kk A(m,kk) B(kk,n) + b[n]
//          m = (n,p,q) output pixel, n = output channel, kk = (r,s,c);
//          A = im2col(x) (contiguous along c), B = W[n][r][s][c].
//   DGRAD  dx[m][c]  = sum_kk A(m,kk) B(kk,c)
//          the input gradient needs W only.  A strided convolution is split
//          into stride_h*stride_w phases (sub-pixel decomposition): the input
//          pixels h with (h + pad_h) mod stride_h = phi_h are reached only by
//          taps r = phi_h + t*stride_h, at output row p = i + delta_h - t for
//          h = h0 + i*stride_h.  Each phase is a dense GEMM (grid z) with no
//          zero-inserted work.  m = (n,i,j), kk = (t_r, t_s, k);
//          A = dy[n][p][q][k] (contiguous along k), B = W[k][r][s][c]
//          (contiguous along c).
//   WGRAD  dW[k][(r,s,c)] = sum_{(n,p,q)} dy[n,p,q][k] * x[n, p*sh-ph+r, q*sw-pw+s][c]
//          the weight gradient needs x only.  Long reductions are split over
//          grid z into fp32 partials, summed by splitk_reduce.
//
// The fully-connected layer is the 1x1 / stride 1 / pad 0 case (UNIT).
//
// Block: 256 threads = 4 waves in a 2x2 grid; block tile BM x BN, K step BK,
// two LDS stages (global loads of tile k+1 overlap the MFMAs of tile k).
// LDS holds both operands as [row][k] (k contiguous, padded rows) so each
// lane fetches its MFMA fragment with one 16-byte LDS read.  Operands that
// are contiguous along k in HBM are copied with 16-byte vectors; operands
// contiguous along m/n are transposed on their way into LDS.
#include "common.h"
#include "../device.h"

namespace ms {

// bf16 fast path (gemm_bf16.hip); each returns -1 when it does not apply.
namespace g2 {
size_t fwd_workspace(const ConvGeom &g);
int conv_fwd(const ConvGeom &g, const void *x, const void *w, const void *bias, void *y, void *ws, hipStream_t st);
size_t dgrad_workspace(const ConvGeom &g, bool with_db);
int conv_dgrad(const ConvGeom &g, const void *dy, const void *w, const void *bias, void *dx, void *ws,
               hipStream_t st, void *db, bool *db_done);
bool wgrad_applies(const ConvGeom &g);
size_t wgrad_workspace(const ConvGeom &g, bool with_db);
int conv_wgrad(const ConvGeom &g, const void *dy, const void *x, void *dw, void *db, void *ws, hipStream_t st);
}  // namespace g2

enum Mode { kFwd = 0, kDgrad = 1, kWgrad = 2 };

struct IgemmParams {
    const void *a;
    const void *b;
    void *c;
    const void *bias;
    ConvGeom g;
    int M, Ng, Kg;     // GEMM extents (DGRAD: bounds over all phases)
    int ntm, ntn;      // tile counts (DGRAD: bounds over all phases)
    int k_split;       // WGRAD: reduction length per split (multiple of BK)
    int splits;
};

// Per-phase geometry of the strided input gradient.
struct Phase {
    int fh, fw;    // phase (phi_h, phi_w)
    int h0, w0;    // first input row / column of the phase
    int Hp, Wp;    // input rows / columns in the phase
    int Rp, Sp;    // taps in the phase
    int dh, dw;    // output-row offset: p = i + dh - t
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

template <typename T, int MODE, int BM, int BN, int BK, bool VEC_OK, bool UNIT>
struct Igemm {
    static constexpr int NT = 256;
    static constexpr int VEC = 16 / sizeof(T);
    static constexpr bool IS_BF16 = sizeof(T) == 2;
    static constexpr int KI = IS_BF16 ? 32 : 4;     // MFMA k per instruction
    static constexpr int KL = KI / 4;               // k elements per lane per fragment
    static constexpr int PADK = IS_BF16 ? 8 : 4;
    static constexpr int LDK = BK + PADK;           // LDS row pitch (elements)
    static constexpr int WM = BM / 2, WN = BN / 2;  // wave tile
    static constexpr int TM = WM / 16, TN = WN / 16;
    // K-contiguous operand: VPR vectors per row
    static constexpr int VPR = BK / VEC;
    // M/N-contiguous operand: vectors per k-row
    static constexpr int VPKA = BM / VEC, VPKB = BN / VEC;
    static constexpr bool A_KC = MODE != kWgrad;    // A contiguous along k
    static constexpr bool B_KC = MODE == kFwd;      // B contiguous along k
    static constexpr int NVA = BM * BK / VEC / NT;
    static constexpr int NVB = BN * BK / VEC / NT;
    static_assert(NVA >= 1 && NVB >= 1, "tile too small for 256 threads");
    static_assert(NT % VPR == 0 && NT % VPKA == 0 && NT % VPKB == 0, "thread map");
    static_assert(BK % KI == 0, "BK must be a multiple of the MFMA k");
};

// BIAS (DGRAD only): add bias[c] to the input gradient -- the forward of a
// transposed convolution; a variant of its own so that the plain input
// gradient keeps its register budget.
template <typename T, int MODE, int BM, int BN, int BK, bool VEC_OK, bool UNIT, bool BIAS = false>
__global__ __launch_bounds__(256) void igemm_kernel(IgemmParams prm) {
    using G = Igemm<T, MODE, BM, BN, BK, VEC_OK, UNIT>;
    constexpr int VEC = G::VEC, LDK = G::LDK, NVA = G::NVA, NVB = G::NVB;
    constexpr int TM = G::TM, TN = G::TN, KL = G::KL, KI = G::KI;

    __shared__ __attribute__((aligned(16))) T smem[2][(BM + BN) * LDK];

    const ConvGeom &g = prm.g;
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm0 = (wave >> 1) * G::WM;
    const int wn0 = (wave & 1) * G::WN;

    // ---- problem extents for this block (DGRAD: per phase) ----
    int M = prm.M, Ng = prm.Ng, Kg = prm.Kg;
    int ntm = prm.ntm, ntn = prm.ntn;
    Phase f{};
    int k_begin = 0, k_end = Kg;
    if constexpr (MODE == kDgrad) {
        f = make_phase(g, blockIdx.z);
        M = g.N * f.Hp * f.Wp;
        Kg = f.Rp * f.Sp * g.K;
        k_end = Kg;
        ntm = (M + BM - 1) / BM;
    }
    if constexpr (MODE == kWgrad) {
        k_begin = blockIdx.z * prm.k_split;
        k_end = min(Kg, k_begin + prm.k_split);
    }
    // tile index: XCD-aware remap, then grouped ordering (8 row tiles share
    // each column sweep so B tiles are reused out of L2)
    const int nb = prm.ntm * prm.ntn;
    const int lt = xcd_remap(blockIdx.x, nb);
    int tm, tn;
    {
        const int GM = 8;
        const int per_group = GM * prm.ntn;
        const int gid = lt / per_group;
        const int first = gid * GM;
        const int gsz = min(prm.ntm - first, GM);
        const int r = lt - gid * per_group;
        tm = first + r % gsz;
        tn = r / gsz;
    }
    if (tm >= ntm || tn >= ntn) return;   // DGRAD phase smaller than the bound
    const int m0 = tm * BM, n0 = tn * BN;

    const T *__restrict__ Ap = static_cast<const T *>(prm.a);
    const T *__restrict__ Bp = static_cast<const T *>(prm.b);

    // ---- per-thread operand coordinates, fixed over the k loop ----
    // A contiguous along k: thread owns rows a_row[i], k-vector a_kv.
    // A contiguous along m: thread owns m-vector a_mv, k-rows a_krow[i].
    const int a_kv = tid % G::VPR;
    const int a_mv = tid % G::VPKA;
    const int b_kv = tid % G::VPR;
    const int b_mv = tid % G::VPKB;

    // A row state
    int a_base[NVA];   // element offset of the row's pixel/sample base
    int a_y[NVA], a_x[NVA];
    bool a_ok[NVA];
    if constexpr (G::A_KC) {
#pragma unroll
        for (int i = 0; i < NVA; ++i) {
            const int row = tid / G::VPR + i * (256 / G::VPR);
            const int m = m0 + row;
            a_ok[i] = m < M;
            const int mm = a_ok[i] ? m : 0;
            if constexpr (UNIT) {
                a_base[i] = mm * (MODE == kFwd ? g.C : g.K);
                a_y[i] = a_x[i] = 0;
            } else if constexpr (MODE == kFwd) {
                const int PQ = g.P * g.Q;
                const int n = mm / PQ, pq = mm - n * PQ;
                const int p = pq / g.Q, q = pq - p * g.Q;
                a_base[i] = n * g.H * g.W * g.C;
                a_y[i] = p * g.sh - g.ph;
                a_x[i] = q * g.sw - g.pw;
            } else {  // DGRAD
                const int HW = f.Hp * f.Wp;
                const int n = HW > 0 ? mm / HW : 0, ij = mm - n * HW;
                const int i2 = f.Wp > 0 ? ij / f.Wp : 0, j2 = ij - i2 * f.Wp;
                a_base[i] = n * g.P * g.Q * g.K;
                a_y[i] = i2 + f.dh;
                a_x[i] = j2 + f.dw;
            }
        }
    }
    // B (contiguous along n) fixed column state for DGRAD / WGRAD
    int b_r = 0, b_s = 0, b_c = 0;
    bool b_colok = true;
    if constexpr (!G::B_KC) {
        const int nn = n0 + b_mv * VEC;
        b_colok = nn < Ng;
        if constexpr (MODE == kWgrad && !UNIT) {
            const int rs = nn / g.C;
            b_c = nn - rs * g.C;
            b_r = rs / g.S;
            b_s = rs - b_r * g.S;
        } else {
            b_c = nn;
        }
    }
    int b_base[NVB];
    bool b_ok[NVB];
    if constexpr (G::B_KC) {  // FWD: rows are output channels
#pragma unroll
        for (int i = 0; i < NVB; ++i) {
            const int row = tid / G::VPR + i * (256 / G::VPR);
            const int n = n0 + row;
            b_ok[i] = n < Ng;
            b_base[i] = (b_ok[i] ? n : 0) * Kg;
        }
    }

    Vec16<T> ra[NVA], rb[NVB];

    // ---- global -> registers ----
    auto load_a = [&](int k0) {
        if constexpr (G::A_KC) {
            if constexpr (VEC_OK) {
                const int kk = k0 + a_kv * VEC;
                const bool kin = kk < k_end;
                int off_k = 0, dy_ = 0, dx_ = 0;
                if constexpr (!UNIT) {
                    if constexpr (MODE == kFwd) {
                        const int rs = kk / g.C, c = kk - rs * g.C;
                        const int r = rs / g.S, s = rs - r * g.S;
                        dy_ = r; dx_ = s; off_k = c;
                    } else {
                        const int t = kk / g.K, k = kk - t * g.K;
                        const int tr = f.Sp > 0 ? t / f.Sp : 0, ts = t - tr * f.Sp;
                        dy_ = -tr; dx_ = -ts; off_k = k;
                    }
                }
#pragma unroll
                for (int i = 0; i < NVA; ++i) {
                    bool ok = kin && a_ok[i];
                    int off;
                    if constexpr (UNIT) {
                        off = a_base[i] + kk;
                    } else if constexpr (MODE == kFwd) {
                        const int ih = a_y[i] + dy_, iw = a_x[i] + dx_;
                        ok = ok && (unsigned)ih < (unsigned)g.H && (unsigned)iw < (unsigned)g.W;
                        off = a_base[i] + (ih * g.W + iw) * g.C + off_k;
                    } else {
                        const int p = a_y[i] + dy_, q = a_x[i] + dx_;
                        ok = ok && (unsigned)p < (unsigned)g.P && (unsigned)q < (unsigned)g.Q;
                        off = a_base[i] + (p * g.Q + q) * g.K + off_k;
                    }
                    ra[i] = ok ? load16(Ap + off) : zero16<T>();
                }
            } else {
                // scalar gather: each element decomposes its own k index
#pragma unroll
                for (int i = 0; i < NVA; ++i) {
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        const int kk = k0 + a_kv * VEC + e;
                        bool ok = a_ok[i] && kk < k_end;
                        int off = 0;
                        if constexpr (UNIT) {
                            off = a_base[i] + kk;
                        } else if constexpr (MODE == kFwd) {
                            const int rs = kk / g.C, c = kk - rs * g.C;
                            const int r = rs / g.S, s = rs - r * g.S;
                            const int ih = a_y[i] + r, iw = a_x[i] + s;
                            ok = ok && (unsigned)ih < (unsigned)g.H && (unsigned)iw < (unsigned)g.W;
                            off = a_base[i] + (ih * g.W + iw) * g.C + c;
                        } else {
                            const int t = kk / g.K, k = kk - t * g.K;
                            const int tr = f.Sp > 0 ? t / f.Sp : 0, ts = t - tr * f.Sp;
                            const int p = a_y[i] - tr, q = a_x[i] - ts;
                            ok = ok && (unsigned)p < (unsigned)g.P && (unsigned)q < (unsigned)g.Q;
                            off = a_base[i] + (p * g.Q + q) * g.K + k;
                        }
                        ra[i].e[e] = ok ? Ap[off] : from_f32<T>(0.f);
                    }
                }
            }
        } else {
            // WGRAD A: A(m = k, kk = npq) = dy[kk][k], contiguous along m
#pragma unroll
            for (int i = 0; i < NVA; ++i) {
                const int kk = k0 + tid / G::VPKA + i * (256 / G::VPKA);
                const int mm = m0 + a_mv * VEC;
                const bool kin = kk < k_end;
                if constexpr (VEC_OK) {
                    ra[i] = (kin && mm < M) ? load16(Ap + kk * g.K + mm) : zero16<T>();
                } else {
#pragma unroll
                    for (int e = 0; e < VEC; ++e)
                        ra[i].e[e] = (kin && mm + e < M) ? Ap[kk * g.K + mm + e] : from_f32<T>(0.f);
                }
            }
        }
    };

    auto load_b = [&](int k0) {
        if constexpr (G::B_KC) {
            // FWD B: W[n][kk], contiguous along kk
#pragma unroll
            for (int i = 0; i < NVB; ++i) {
                const int kk = k0 + b_kv * VEC;
                if constexpr (VEC_OK) {
                    rb[i] = (b_ok[i] && kk < k_end) ? load16(Bp + b_base[i] + kk) : zero16<T>();
                } else {
#pragma unroll
                    for (int e = 0; e < VEC; ++e)
                        rb[i].e[e] = (b_ok[i] && kk + e < k_end) ? Bp[b_base[i] + kk + e] : from_f32<T>(0.f);
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < NVB; ++i) {
                const int kk = k0 + tid / G::VPKB + i * (256 / G::VPKB);
                bool ok = kk < k_end && b_colok;
                int off = 0;
                if constexpr (MODE == kDgrad) {
                    // B(kk = (t_r, t_s, k), c) = W[k][r][s][c]
                    if constexpr (UNIT) {
                        off = kk * g.C + b_c;
                    } else {
                        const int t = kk / g.K, k = kk - t * g.K;
                        const int tr = f.Sp > 0 ? t / f.Sp : 0, ts = t - tr * f.Sp;
                        const int r = f.fh + tr * g.sh, s = f.fw + ts * g.sw;
                        off = ((k * g.R + r) * g.S + s) * g.C + b_c;
                    }
                } else {
                    // WGRAD B(kk = (n,p,q), (r,s,c)) = x[n][p*sh-ph+r][q*sw-pw+s][c]
                    if constexpr (UNIT) {
                        off = kk * g.C + b_c;
                    } else {
                        const int PQ = g.P * g.Q;
                        const int n = kk / PQ, pq = kk - n * PQ;
                        const int p = pq / g.Q, q = pq - p * g.Q;
                        const int ih = p * g.sh - g.ph + b_r, iw = q * g.sw - g.pw + b_s;
                        ok = ok && (unsigned)ih < (unsigned)g.H && (unsigned)iw < (unsigned)g.W;
                        off = ((n * g.H + ih) * g.W + iw) * g.C + b_c;
                    }
                }
                if constexpr (VEC_OK) {
                    rb[i] = ok ? load16(Bp + off) : zero16<T>();
                } else {
                    const int nn = n0 + b_mv * VEC;
#pragma unroll
                    for (int e = 0; e < VEC; ++e) {
                        bool oke = ok && (nn + e) < Ng;
                        int offe = off + e;
                        if constexpr (MODE == kWgrad && !UNIT) {
                            // a vector may cross an (r,s) boundary: decompose each element
                            const int n2 = nn + e;
                            const int rs = n2 / g.C, c = n2 - rs * g.C;
                            const int r = rs / g.S, s = rs - r * g.S;
                            const int PQ = g.P * g.Q;
                            const int n = kk / PQ, pq = kk - n * PQ;
                            const int p = pq / g.Q, q = pq - p * g.Q;
                            const int ih = p * g.sh - g.ph + r, iw = q * g.sw - g.pw + s;
                            oke = kk < k_end && n2 < Ng && (unsigned)ih < (unsigned)g.H &&
                                  (unsigned)iw < (unsigned)g.W;
                            offe = ((n * g.H + ih) * g.W + iw) * g.C + c;
                        }
                        rb[i].e[e] = oke ? Bp[offe] : from_f32<T>(0.f);
                    }
                }
            }
        }
    };

    // ---- registers -> LDS ----
    auto store_lds = [&](int buf) {
        T *As = smem[buf];
        T *Bs = smem[buf] + BM * LDK;
        if constexpr (G::A_KC) {
#pragma unroll
            for (int i = 0; i < NVA; ++i) {
                const int row = tid / G::VPR + i * (256 / G::VPR);
                store16(As + row * LDK + a_kv * VEC, ra[i]);
            }
        } else {
#pragma unroll
            for (int i = 0; i < NVA; ++i) {
                const int kr = tid / G::VPKA + i * (256 / G::VPKA);
#pragma unroll
                for (int e = 0; e < VEC; ++e) As[(a_mv * VEC + e) * LDK + kr] = ra[i].e[e];
            }
        }
        if constexpr (G::B_KC) {
#pragma unroll
            for (int i = 0; i < NVB; ++i) {
                const int row = tid / G::VPR + i * (256 / G::VPR);
                store16(Bs + row * LDK + b_kv * VEC, rb[i]);
            }
        } else {
#pragma unroll
            for (int i = 0; i < NVB; ++i) {
                const int kr = tid / G::VPKB + i * (256 / G::VPKB);
#pragma unroll
                for (int e = 0; e < VEC; ++e) Bs[(b_mv * VEC + e) * LDK + kr] = rb[i].e[e];
            }
        }
    };

    floatx4 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

    const int nk = k_end > k_begin ? (k_end - k_begin + BK - 1) / BK : 0;
    if (nk > 0) {
        load_a(k_begin);
        load_b(k_begin);
        store_lds(0);
    }
    __syncthreads();

    const int fr = lane & 15;         // fragment row/col within a 16x16 tile
    const int fk = (lane >> 4) * KL;  // fragment k offset
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        const bool more = kt + 1 < nk;
        if (more) {
            load_a(k_begin + (kt + 1) * BK);
            load_b(k_begin + (kt + 1) * BK);
        }
        const T *As = smem[buf];
        const T *Bs = smem[buf] + BM * LDK;
#pragma unroll
        for (int kk = 0; kk < BK; kk += KI) {
            if constexpr (G::IS_BF16) {
                bf16x8 af[TM], bfr[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i)
                    af[i] = *reinterpret_cast<const bf16x8 *>(As + (wm0 + i * 16 + fr) * LDK + kk + fk);
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    bfr[j] = *reinterpret_cast<const bf16x8 *>(Bs + (wn0 + j * 16 + fr) * LDK + kk + fk);
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
            } else {
                float af[TM], bfr[TN];
#pragma unroll
                for (int i = 0; i < TM; ++i) af[i] = As[(wm0 + i * 16 + fr) * LDK + kk + fk];
#pragma unroll
                for (int j = 0; j < TN; ++j) bfr[j] = Bs[(wn0 + j * 16 + fr) * LDK + kk + fk];
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i], bfr[j], acc[i][j], 0, 0, 0);
            }
        }
        if (more) store_lds(buf ^ 1);
        __syncthreads();
    }

    // ---- epilogue: lane holds D[4*(lane/16)+v][lane%16] of each 16x16 tile ----
    const int er = (lane >> 4) * 4;
    const int ec = lane & 15;
    if constexpr (MODE == kFwd) {
        T *Y = static_cast<T *>(prm.c);
        const T *bias = static_cast<const T *>(prm.bias);
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int n = n0 + wn0 + j * 16 + ec;
            if (n >= Ng) continue;
            const float bv = bias ? to_f32(bias[n]) : 0.f;
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int m = m0 + wm0 + i * 16 + er + v;
                    if (m < M) Y[m * Ng + n] = from_f32<T>(acc[i][j][v] + bv);
                }
        }
    } else if constexpr (MODE == kDgrad) {
        T *DX = static_cast<T *>(prm.c);
        const T *bias = static_cast<const T *>(prm.bias);
        const int HW = f.Hp * f.Wp;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int m = m0 + wm0 + i * 16 + er + v;
                if (m >= M) continue;
                int pix;
                if constexpr (UNIT) {
                    pix = m;
                } else {
                    const int n = m / HW, ij = m - n * HW;
                    const int i2 = ij / f.Wp, j2 = ij - i2 * f.Wp;
                    pix = (n * g.H + f.h0 + i2 * g.sh) * g.W + f.w0 + j2 * g.sw;
                }
#pragma unroll
                for (int j = 0; j < TN; ++j) {
                    const int c = n0 + wn0 + j * 16 + ec;
                    if (c >= Ng) continue;
                    if constexpr (BIAS) DX[pix * g.C + c] = from_f32<T>(acc[i][j][v] + to_f32(bias[c]));
                    else DX[pix * g.C + c] = from_f32<T>(acc[i][j][v]);
                }
            }
    } else {
        const bool partial = prm.splits > 1;
        T *DW = static_cast<T *>(prm.c);
        float *WS = static_cast<float *>(prm.c) + (size_t)blockIdx.z * M * Ng;
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int n = n0 + wn0 + j * 16 + ec;
            if (n >= Ng) continue;
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int m = m0 + wm0 + i * 16 + er + v;
                    if (m >= M) continue;
                    if (partial) WS[m * Ng + n] = acc[i][j][v];
                    else DW[m * Ng + n] = from_f32<T>(acc[i][j][v]);
                }
        }
    }
}

// out[i] = sum_z ws[z][i], rounded once to T.
template <typename T>
__global__ __launch_bounds__(256) void splitk_reduce_kernel(const float *__restrict__ ws, int splits,
                                                            int64_t n, T *__restrict__ out) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x * 4;
    for (int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4; i < n; i += stride) {
        if ((n & 3) == 0) {   // every slice z*n + i is 16-byte aligned
            floatx4 s = *reinterpret_cast<const floatx4 *>(ws + i);
            for (int z = 1; z < splits; ++z) {
                floatx4 t = *reinterpret_cast<const floatx4 *>(ws + (int64_t)z * n + i);
                s += t;
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) out[i + e] = from_f32<T>(s[e]);
        } else {
            for (int64_t k = i; k < n && k < i + 4; ++k) {
                float s = 0.f;
                for (int z = 0; z < splits; ++z) s += ws[(int64_t)z * n + k];
                out[k] = from_f32<T>(s);
            }
        }
    }
}

// ------------------------------------------------------------------ launchers
namespace {

constexpr int kBM = 128, kBN = 128;
template <typename T> constexpr int bk_of() { return sizeof(T) == 2 ? 32 : 16; }

bool aligned16(const void *p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

bool is_unit(const ConvGeom &g) {
    return g.R == 1 && g.S == 1 && g.sh == 1 && g.sw == 1 && g.ph == 0 && g.pw == 0 &&
           g.P == g.H && g.Q == g.W;
}

template <typename T, int MODE, bool VEC_OK, bool UNIT>
int launch_t(const IgemmParams &prm, dim3 grid, hipStream_t st) {
    constexpr int BK = bk_of<T>();
    const unsigned pk = MODE == kFwd ? kProfFwd : MODE == kDgrad ? kProfDgrad : kProfWgrad;
    prof_mark(pk, st, true);
    if (MODE == kDgrad && prm.bias)
        hipLaunchKernelGGL((igemm_kernel<T, MODE, kBM, kBN, BK, VEC_OK, UNIT, MODE == kDgrad>), grid, dim3(256), 0, st,
                           prm);
    else
        hipLaunchKernelGGL((igemm_kernel<T, MODE, kBM, kBN, BK, VEC_OK, UNIT>), grid, dim3(256), 0, st, prm);
    const int err = (int)hipGetLastError();
    prof_mark(pk, st, false);
    return err;
}

template <typename T, int MODE>
int launch_mode(const IgemmParams &prm, dim3 grid, bool vec_ok, bool unit, hipStream_t st) {
    if (vec_ok) {
        return unit ? launch_t<T, MODE, true, true>(prm, grid, st)
                    : launch_t<T, MODE, true, false>(prm, grid, st);
    }
    return unit ? launch_t<T, MODE, false, true>(prm, grid, st)
                : launch_t<T, MODE, false, false>(prm, grid, st);
}

template <int MODE>
int launch_dtype(int dtype, const IgemmParams &prm, dim3 grid, bool vec_ok, bool unit, hipStream_t st) {
    if (dtype == kBF16) return launch_mode<bf16, MODE>(prm, grid, vec_ok, unit, st);
    return launch_mode<float, MODE>(prm, grid, vec_ok, unit, st);
}

int vec_elems(int dtype) { return dtype == kBF16 ? 8 : 4; }

struct SplitPlan {
    int splits, k_split;
};

SplitPlan wgrad_split(int dtype, const ConvGeom &g) {
    const int M = g.K, Ng = g.R * g.S * g.C, Kg = g.N * g.P * g.Q;
    const int BK = dtype == kBF16 ? 32 : 16;
    const int tiles = ((M + kBM - 1) / kBM) * ((Ng + kBN - 1) / kBN);
    int splits = 1;
    const int target = 512;  // ~2 blocks per CU
    if (tiles < target && Kg >= 8 * BK) {
        splits = (target + tiles - 1) / tiles;
        splits = std::min(splits, Kg / (4 * BK));
        splits = std::max(splits, 1);
    }
    if (Kg == 0) return {1, BK};   // empty reduction: one split writes zeros
    int k_split = (Kg + splits - 1) / splits;
    k_split = (k_split + BK - 1) / BK * BK;
    splits = (Kg + k_split - 1) / k_split;
    return {splits, k_split};
}

}  // namespace

size_t conv_fwd_workspace(int dtype, const ConvGeom &g) {
    return dtype == kBF16 ? g2::fwd_workspace(g) : 0;
}

int launch_conv_fwd(int dtype, const ConvGeom &g, const void *x, const void *w, const void *bias,
                    void *y, void *ws, void *stream) {
    if (dtype == kBF16) {
        const int r = g2::conv_fwd(g, x, w, bias, y, ws, (hipStream_t)stream);
        if (r >= 0) return r;
    }
    IgemmParams prm{};
    prm.a = x; prm.b = w; prm.c = y; prm.bias = bias; prm.g = g;
    prm.M = g.N * g.P * g.Q;
    prm.Ng = g.K;
    prm.Kg = g.R * g.S * g.C;
    prm.ntm = (prm.M + kBM - 1) / kBM;
    prm.ntn = (prm.Ng + kBN - 1) / kBN;
    prm.splits = 1;
    prm.k_split = prm.Kg;
    if (prm.M == 0 || prm.Ng == 0) return 0;
    const int V = vec_elems(dtype);
    const bool vec_ok = g.C % V == 0 && aligned16(x) && aligned16(w);
    dim3 grid(prm.ntm * prm.ntn, 1, 1);
    return launch_dtype<kFwd>(dtype, prm, grid, vec_ok, is_unit(g), (hipStream_t)stream);
}

size_t conv_dgrad_workspace(int dtype, const ConvGeom &g, bool with_db) {
    return dtype == kBF16 ? g2::dgrad_workspace(g, with_db) : 0;
}

int launch_conv_dgrad(int dtype, const ConvGeom &g, const void *dy, const void *w, const void *bias,
                      void *dx, void *ws, void *stream, void *db, bool *db_done) {
    if (db_done) *db_done = false;
    if (dtype == kBF16) {
        const int r = g2::conv_dgrad(g, dy, w, bias, dx, ws, (hipStream_t)stream, db, db_done);
        if (r >= 0) return r;
    }
    IgemmParams prm{};
    prm.a = dy; prm.b = w; prm.c = dx; prm.bias = bias; prm.g = g;
    // bounds over phases: ceil(H / sh) rows, ceil(R / sh) taps
    const int Hb = (g.H + g.sh - 1) / g.sh, Wb = (g.W + g.sw - 1) / g.sw;
    prm.M = g.N * Hb * Wb;
    prm.Ng = g.C;
    prm.Kg = ((g.R + g.sh - 1) / g.sh) * ((g.S + g.sw - 1) / g.sw) * g.K;
    prm.ntm = (prm.M + kBM - 1) / kBM;
    prm.ntn = (prm.Ng + kBN - 1) / kBN;
    prm.splits = 1;
    if (prm.M == 0 || prm.Ng == 0) return 0;
    const int V = vec_elems(dtype);
    const bool vec_ok = g.K % V == 0 && g.C % V == 0 && aligned16(dy) && aligned16(w);
    dim3 grid(prm.ntm * prm.ntn, 1, g.sh * g.sw);
    return launch_dtype<kDgrad>(dtype, prm, grid, vec_ok, is_unit(g), (hipStream_t)stream);
}

size_t conv_wgrad_workspace(int dtype, const ConvGeom &g, bool with_db) {
    // the fallback below may run when the fast path turns out not to apply
    // (pointer alignment), so the workspace covers both
    SplitPlan sp = wgrad_split(dtype, g);
    const size_t v1 = sp.splits <= 1 ? 0 : (size_t)sp.splits * (size_t)g.K * (size_t)(g.R * g.S * g.C) * sizeof(float);
    if (dtype == kBF16 && g2::wgrad_applies(g)) return std::max(v1, g2::wgrad_workspace(g, with_db));
    return v1;
}

int launch_conv_wgrad(int dtype, const ConvGeom &g, const void *dy, const void *x, void *dw,
                      void *db, void *ws, void *stream, bool *db_done) {
    hipStream_t st = (hipStream_t)stream;
    *db_done = false;
    if (dtype == kBF16) {
        const int r = g2::conv_wgrad(g, dy, x, dw, db, ws, st);
        if (r >= 0) {
            *db_done = db != nullptr;
            return r;
        }
    }
    SplitPlan sp = wgrad_split(dtype, g);
    IgemmParams prm{};
    prm.a = dy; prm.b = x; prm.g = g;
    prm.M = g.K;
    prm.Ng = g.R * g.S * g.C;
    prm.Kg = g.N * g.P * g.Q;
    prm.ntm = (prm.M + kBM - 1) / kBM;
    prm.ntn = (prm.Ng + kBN - 1) / kBN;
    prm.splits = sp.splits;
    prm.k_split = sp.k_split;
    prm.c = sp.splits > 1 ? ws : dw;
    if (prm.M == 0 || prm.Ng == 0) return 0;
    const int V = vec_elems(dtype);
    const bool vec_ok = g.K % V == 0 && g.C % V == 0 && aligned16(dy) && aligned16(x);
    dim3 grid(prm.ntm * prm.ntn, 1, sp.splits);
    int err = launch_dtype<kWgrad>(dtype, prm, grid, vec_ok, is_unit(g), st);
    if (err || sp.splits <= 1) return err;
    const int64_t n = (int64_t)prm.M * prm.Ng;
    const int blocks = (int)std::min<int64_t>((n / 4 + 255) / 256 + 1, 4096);
    if (dtype == kBF16)
        hipLaunchKernelGGL(splitk_reduce_kernel<bf16>, dim3(blocks), dim3(256), 0, st,
                           (const float *)ws, sp.splits, n, (bf16 *)dw);
    else
        hipLaunchKernelGGL(splitk_reduce_kernel<float>, dim3(blocks), dim3(256), 0, st,
                           (const float *)ws, sp.splits, n, (float *)dw);
    return (int)hipGetLastError();
}

}  // namespace ms
