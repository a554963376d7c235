// na_fwd.hip -- fused neighborhood-attention forward for gfx950.
//
// Fused NA (Sec. 3.3, Fig. "fna-vis"): queries are tiled in their own 1-D /
// 2-D / 3-D layout; the key/value tile is the halo that covers every
// neighbourhood of the query tile; scores go through the NA mask and an online
// softmax (Sec. 2) and straight into the product with V.  Only the output and
// the per-query logsumexp are written.  Dilation is handled as extra
// workgroups over the sub-lattices x = g (mod d) (Sec. 3.4).
//
// MI355X mapping:
//   * workgroup = W waves (4; 8 for large 1-D problems) = one query tile of
//     one (batch, head, dilation group); each wave owns QM x 16 queries of it
//     (a sub-box);
//   * the workgroup's key halo is cut into blocks of 16 keys that run along
//     the innermost axis; stages of SB blocks go straight from HBM to LDS
//     (16-byte direct-to-LDS loads, double buffered when there is more than
//     one stage), K and V both as swizzled unpadded rows; V^T fragments are
//     gathered with the transposed LDS read, so no transposed copy exists;
//   * a wave only runs the matrix cores on blocks that intersect its own
//     sub-box halo, and evaluates the mask only on blocks that are not inside
//     every one of its windows;
//   * S^T = K Q^T (16 keys x 16 queries per MFMA) leaves each query's scores
//     in one lane column; the row maximum needs two lane-swap steps, and P^T
//     feeds O^T = V^T P^T directly as the B operand;
//   * scores are scaled once into base 2 (so the row maximum maps to exactly
//     exp2(0) = 1 and a window of one key returns V bit for bit); the running
//     maximum is only raised (and O rescaled) when a row's maximum grows by
//     more than kLazy, which keeps every P <= 2^kLazy.  Each lane tests its
//     own share of a row against the threshold; the cross-lane row maximum is
//     formed only in the (rare) raising branch;
//   * with one query block per wave, 16-bit types sum each row of the rounded
//     P on the matrix cores: one more MFMA with an all-ones V^T block leaves
//     the full row sum in every lane (with two blocks the extra accumulators
//     would cost a wave of occupancy, so those sum with v_dot2).
#include <algorithm>
#include <cmath>
#include <type_traits>

#include "na_launch.h"
#include "na_stage.h"

namespace na {

constexpr float kLazy = 8.f;  // base-2 headroom before the running max is raised

template <int R, int D, typename T, int QM, int SB, int W = 4>
struct FwdCfg {
    static constexpr int kWaves = W;
    static constexpr int kThreads = W * kWave;
    static constexpr int kKeys = SB * 16;  // keys per stage
    static constexpr int kTileBytes = kKeys * Rows<T, D>::kRowBytes;
    static constexpr size_t kBufBytes = 2 * kTileBytes;  // K rows, then V rows
    static constexpr int kKS = D / 32;  // contraction steps over D
    static constexpr int kDB = D / 16;  // 16-wide blocks of D
    using Ld = DirectRows<T, D, kKeys, W, (R > 1)>;
    static_assert(SB % 2 == 0 && SB <= 32, "stage blocks are tested by one lane each");
};

// Workgroups per CU the register allocation must allow: four waves per SIMD
// for the 16-bit kernels that fit 128 VGPRs (every one at D <= 64, and the
// one-block ones at D = 128); the others take what they need.
template <int D, typename T, int QM, int W>
constexpr int fwd_min_blocks() {
    return sizeof(T) == 2 && (D <= 64 || QM == 1) ? 16 / W : 1;
}

// c = scale * log2(e): scores are kept in base 2.  SHORT = 1: every halo row
// holds at most two 16-key blocks (rank >= 2), so the inner-axis mask is a
// per-lane constant; SHORT = 0: general masking with mask-free full blocks.
template <int R, int D, typename T, int QM, int SB, int SHORT, int W>
__global__ __launch_bounds__(W * kWave, (fwd_min_blocks<D, T, QM, W>())) void na_fwd_kernel(
    Geo g, const T* __restrict__ qg, const T* __restrict__ kg, const T* __restrict__ vg,
    T* __restrict__ og, float* __restrict__ lseg, float c) {
    using C = FwdCfg<R, D, T, QM, SB, W>;
    using x8 = typename Tr<T>::x8;
    extern __shared__ __align__(16) unsigned char smem_raw[];

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    // (masked: the launch has W waves, which lets the compiler drop the
    // staging loops' bounds tests)
    const int wave = uniform((tid >> 6) & (W - 1));
    const int col = lane & 15;  // query column of this lane
    const int grp = lane >> 4;  // 16-lane group

    // ---- workgroup -> (bh, dilation group, tile) ----
    fetch_geo<R>(g);
    asm volatile("" ::"s"(qg), "s"(kg), "s"(vg), "s"(og), "s"(lseg), "s"(c));
    const int bid = xcd_remap(blockIdx.x, g.nwg);
    int bh, gc[kMaxRank], tc[kMaxRank], n[kMaxRank], to[kMaxRank];
    decode_workgroup<R>(g, bid, bh, gc, tc, n);

    Box<R> halo;
#pragma unroll
    for (int a = 0; a < R; ++a) {
        to[a] = tc[a] * g.T[a];
        if (to[a] >= n[a]) return;  // tile beyond this (shorter) group: uniform exit
        const int last = min(to[a] + g.T[a], n[a]) - 1;
        const bool ca = g.causal[a] != 0;
        halo.lo[a] = win_start(to[a], n[a], g.k[a], ca);
        halo.E[a] = win_last(last, n[a], g.k[a], ca) + 1 - halo.lo[a];
    }
    halo.finish(g, gc);

    const size_t slice = (size_t)bh * g.N * D;
    const T* kb = kg + slice;
    const T* vb = vg + slice;
    const int tstep = g.d[R - 1];  // token step along the innermost axis

    // ---- staging: K and V rows straight to LDS, one address set for both ----
    // The first stage is issued as soon as the halo is known, so that its
    // loads are in flight during the per-wave and per-lane set-up below.
    typename C::Ld ld;
    auto issue_stage = [&](int s, int buf) {
        ld.compute(halo, s * SB, tstep, wave, lane);
        unsigned char* tile = smem_raw + buf * C::kBufBytes;
        ld.issue(kb, tile, wave);
        ld.issue(vb, tile + C::kTileBytes, wave);
    };
    issue_stage(0, 0);

    // ---- this wave's query sub-box: its halo and the keys inside all of its windows ----
    int wc[kMaxRank], wo[kMaxRank];
    unravel_pow2<R>(wave, g.lgWGd, wc);
    bool wave_live = true;
    WaveRange<R> wr;
#pragma unroll
    for (int a = 0; a < R; ++a) {
        wo[a] = to[a] + wc[a] * g.WT[a];
        if (wo[a] >= n[a]) wave_live = false;
        const int f = min(wo[a], n[a] - 1);
        const int l = min(wo[a] + g.WT[a], n[a]) - 1;
        const bool ca = g.causal[a] != 0;
        const int sf = win_start(f, n[a], g.k[a], ca), sl = win_start(l, n[a], g.k[a], ca);
        const int ef = win_last(f, n[a], g.k[a], ca), el = win_last(l, n[a], g.k[a], ca);
        wr.set(a, sf - halo.lo[a], el + 1 - halo.lo[a], sl - halo.lo[a], ef + 1 - halo.lo[a]);
    }

    // ---- per-lane queries: validity, window starts (relative to the halo), Q ----
    int qs[QM][kMaxRank];
    bool qvalid[QM];
    size_t qoff[QM];
    x8 qf[QM][C::kKS];
#pragma unroll
    for (int m = 0; m < QM; ++m) {
        int cc[kMaxRank];
        unravel_pow2<R>(m * 16 + col, g.lgWT, cc);
        bool ok = wave_live;
        int tok = 0;
#pragma unroll
        for (int a = 0; a < R; ++a) {
            int p = wo[a] + cc[a];
            if (p >= n[a]) ok = false;
            p = min(p, n[a] - 1);
            qs[m][a] = mask_start(p, n[a], g.k[a], g.causal[a] != 0) - halo.lo[a];
            tok += (gc[a] + g.d[a] * p) * g.ts[a];
        }
        qvalid[m] = ok;
        qoff[m] = slice + (size_t)tok * D;
#pragma unroll
        // unconditional: qoff points at a real (clamped) query even for absent
        // slots, whose results are discarded; no wait before the K/V loads
        for (int s = 0; s < C::kKS; ++s) qf[m][s] = ld_x8<T>(qg + qoff[m] + s * 32 + grp * 8);
    }

    RowFrag<T, D> kfr;
    ColFrag<T, D> vfr;
    kfr.init(lane);
    vfr.init(lane);

    // ---- online-softmax state (per lane: its query column) ----
    // mref: running reference (base 2, -inf until the row sees a key);
    // negm = -mref (0 while mref = -inf) is the scores' addend and thr the
    // score above which the reference must be raised.
    // Row sums: with kMfmaSum, lsum[m] accumulates ones^T P^T on the matrix
    // cores (every entry is the row sum); otherwise each lane sums its share
    // of P in lrow[m], reduced across the four lane groups at the end.
    // Two blocks per wave: the matrix cores at D = 32, and in 1-D at D = 64,
    // where the two extra accumulators leave the occupancy as it is
    // (elsewhere they cost a wave per SIMD).
    constexpr bool kMfmaSum = sizeof(T) == 2 && (QM == 1 || D <= 32 || (R == 1 && D <= 64));
    // Score addends folded into the accumulators.  Not for D = 128 (the
    // addend vectors would cost it occupancy) nor bf16 (rounding c*Q to 8
    // mantissa bits would add an error comparable to that of P itself).
    constexpr bool kFoldAdd = D <= 64 && !std::is_same_v<T, __bf16>;
    x8 ones;
#pragma unroll
    for (int j = 0; j < 8; ++j) ones[j] = (T)1.0f;
    // kept in four registers for the whole loop: rebuilt from the constant
    // it would cost three moves per tile
    if constexpr (kMfmaSum) {
        i32x4 u = __builtin_bit_cast(i32x4, ones);
        asm volatile("" : "+v"(u));
        ones = __builtin_bit_cast(x8, u);
    }
    f32x4 oacc[QM][C::kDB], lsum[QM];
    float mref[QM], negm[QM], thr[QM], lrow[QM];
    // kFoldAdd: negm in all four slots, the accumulator seed of full tiles,
    // kept as a vector so the matrix cores read it in place (no per-tile splat)
    f32x4 negm4[QM];
#pragma unroll
    for (int m = 0; m < QM; ++m) {
        mref[m] = -INFINITY;
        negm[m] = 0.f;
        negm4[m] = f32x4{0.f, 0.f, 0.f, 0.f};
        thr[m] = -INFINITY;
        lsum[m] = f32x4{0.f, 0.f, 0.f, 0.f};
        lrow[m] = 0.f;
#pragma unroll
        for (int db = 0; db < C::kDB; ++db) oacc[m][db] = f32x4{0.f, 0.f, 0.f, 0.f};
    }
    // Halo rows of at most two 16-key blocks (the usual 2-D / 3-D case): the
    // inner-axis test of this lane's 4 key slots is fixed for the whole
    // kernel, so it is folded into per-slot FMA addends (negm where valid,
    // -inf where not), refreshed only when the reference moves.  Block bi of
    // a tile has inner block index bi when rows hold two blocks, else 0.
    constexpr bool short_rows = SHORT != 0 && R > 1;
    f32x4 ain[QM][2];
    auto refresh_addends = [&](int m) {
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int ib = halo.nbr == 2 ? bi : 0;
                const bool v =
                    (unsigned)(ib * 16 + grp * 4 + r - qs[m][R - 1]) < (unsigned)g.k[R - 1];
                ain[m][bi][r] = v ? negm[m] : -INFINITY;
            }
    };
    if (R > 1) {
#pragma unroll
        for (int m = 0; m < QM; ++m) refresh_addends(m);
    }

    const int nst = (halo.nb + SB - 1) / SB;
    wait_vmem();
    __syncthreads();
    // kFoldAdd: Q scaled once by c = scale*log2(e) and rounded to T, so the
    // matrix cores produce base-2 scores (after the wait: the loads above are
    // in flight together)
    if constexpr (kFoldAdd)
#pragma unroll
    for (int m = 0; m < QM; ++m)
#pragma unroll
        for (int st = 0; st < C::kKS; ++st)
#pragma unroll
            for (int j = 0; j < 8; ++j) qf[m][st][j] = Tr<T>::cvt((float)qf[m][st][j] * c);

    ChunkTests<R, SB> ct;  // this wave's block tests, 64 blocks at a time
    for (int s = 0; s < nst; ++s) {
        if (s + 1 < nst) issue_stage(s + 1, (s + 1) & 1);
        const unsigned char* ks = smem_raw + (s & 1) * C::kBufBytes;
        const unsigned char* vs = ks + C::kTileBytes;

        if (wave_live) {
            // the halo's blocks are tested against this wave's queries (one
            // block per lane, 64 at a time); the wave then visits only the
            // tiles (block pairs) with a relevant block, reading their
            // coordinates back from the lanes
            ct.stage(wr, halo, s, lane);
            const uint64_t relm = ct.rel_bits();
            const uint64_t fullm = ct.full_bits();
            const uint64_t ofullm = ct.ofull_bits();
            uint64_t tiles = (relm | (relm >> 1)) & 0x5555555555555555ull;
            // The body of one tile (block pair tp), by kind: 0 general; 1 both
            // blocks inside every window of the wave's queries (no mask); 2 short
            // rows, both blocks inside every window along the outer axes (the
            // mask is the per-lane inner-axis addend alone, used in place); 3 / 4
            // short rows, only the first / second block so.
            auto tile = [&](int tp, auto tile_kind) {
                constexpr int kKind = decltype(tile_kind)::value;
                constexpr bool kFull = kKind == 1;
                // block bi inside every window along the outer axes
                constexpr bool kOF[2] = {kKind == 2 || kKind == 3, kKind == 2 || kKind == 4};
                bool rel[2], full[2];
                int boc[2][kMaxRank], bin0[2];
#pragma unroll
                for (int bi = 0; bi < 2; ++bi) {
                    const int j = tp * 2 + bi;
                    rel[bi] = kFull || kOF[bi] || ((relm >> j) & 1);
                    full[bi] = kFull || ((fullm >> j) & 1);
                    bin0[bi] = ct.inner0(j);
#pragma unroll
                    for (int a = 0; a < R - 1; ++a) boc[bi][a] = ct.outer(j, a);
                }

                // ---- S^T = K Q^T for both blocks ----
                // Both blocks are read and multiplied without a branch: a block
                // outside this wave's halo is masked below, and every row of
                // the stage buffer holds finite data (missing keys are
                // stand-in rows).  The V fragments of the tile are read here
                // too (D = 32), so one LDS round trip serves the whole tile.
                constexpr int kRowB = Rows<T, D>::kRowBytes;
                x8 kf[2][C::kKS];
#pragma unroll
                for (int bi = 0; bi < 2; ++bi)
#pragma unroll
                    for (int st = 0; st < C::kKS; ++st)
                        kf[bi][st] = kfr.read(ks + (tp * 2 + bi) * 16 * kRowB, st);
                constexpr bool kEarlyV = D == 32;
                x8 vf[C::kDB];
                auto read_v = [&]() {
#pragma unroll
                    for (int db = 0; db < C::kDB; ++db)
                        vf[db] = vfr.read(vs + tp * 32 * kRowB, db, lane);
                };
                if (kEarlyV) read_v();
                // ---- Y^T = c K Q^T + A, A the addend: -m on valid pairs, -inf on masked ----
                // (base 2, relative to the running reference m).  With kFoldAdd the
                // accumulator starts at A and Q is prescaled, so the matrix cores
                // produce Y; otherwise one FMA per score applies c and A.
                auto score_addend = [&](int m, int bi) {
                    f32x4 add;
                    if (!short_rows && full[bi]) {
                        add = f32x4{negm[m], negm[m], negm[m], negm[m]};
                    } else {
                        bool outer_ok = rel[bi];
                        if (!kOF[bi]) {
#pragma unroll
                            for (int a = 0; a < R - 1; ++a)
                                outer_ok = outer_ok &&
                                           (unsigned)(boc[bi][a] - qs[m][a]) < (unsigned)g.k[a];
                        }
                        // generic rows: slot r is valid when base + r lies in [0, lim),
                        // lim folding the outer axes in (0 fails every slot)
                        const int base = bin0[bi] + grp * 4 - qs[m][R - 1];
                        const unsigned lim = outer_ok ? (unsigned)g.k[R - 1] : 0u;
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            add[r] = short_rows ? (outer_ok ? ain[m][bi][r] : -INFINITY)
                                     : (unsigned)(base + r) < lim ? negm[m] : -INFINITY;
                    }
                    return add;
                };
                f32x4 sacc[QM][2];
#pragma unroll
                for (int bi = 0; bi < 2; ++bi)
#pragma unroll
                    for (int m = 0; m < QM; ++m) {
                        // (the first product of a full tile reads negm4 in place, of an
                        // outer-full tile of short rows the inner addends)
                        if (kFoldAdd && !short_rows && full[bi])
                            sacc[m][bi] = Tr<T>::mma(kf[bi][0], qf[m][0], negm4[m]);
                        else if (kFoldAdd && short_rows && kOF[bi])
                            sacc[m][bi] = Tr<T>::mma(kf[bi][0], qf[m][0], ain[m][bi]);
                        else
                            sacc[m][bi] = Tr<T>::mma(kf[bi][0], qf[m][0],
                                                     kFoldAdd ? score_addend(m, bi)
                                                              : f32x4{0.f, 0.f, 0.f, 0.f});
#pragma unroll
                        for (int st = 1; st < C::kKS; ++st)
                            sacc[m][bi] = Tr<T>::mma(kf[bi][st], qf[m][st], sacc[m][bi]);
                    }

                // ---- online softmax per query block ----
                x8 pf[QM];
#pragma unroll
                for (int m = 0; m < QM; ++m) {
                    float y[2][4];
#pragma unroll
                    for (int bi = 0; bi < 2; ++bi) {
                        if constexpr (kFoldAdd) {
#pragma unroll
                            for (int r = 0; r < 4; ++r) y[bi][r] = sacc[m][bi][r];
                        } else {
                            const f32x4 add = score_addend(m, bi);
#pragma unroll
                            for (int r = 0; r < 4; ++r) y[bi][r] = fmaf(sacc[m][bi][r], c, add[r]);
                        }
                    }
                    // this lane's share of the row; the row maximum exceeds the
                    // threshold exactly when some lane's share does
                    // (a chain, so that it becomes three v_max3 and one v_max)
                    const float lmax = fmaxf(
                        fmaxf(fmaxf(fmaxf(fmaxf(fmaxf(fmaxf(y[0][0], y[0][1]), y[0][2]), y[0][3]),
                                          y[1][0]),
                                    y[1][1]),
                              y[1][2]),
                        y[1][3]);
                    // raise the reference on the first valid key of a row, or when
                    // the row grows by more than kLazy (rare, wave-uniform branch)
                    if (__builtin_amdgcn_ballot_w64(lmax > thr[m])) {
                        const float ymax = group_max4(lmax);
                        const bool raise = ymax > thr[m];
                        const float dlt = raise ? ymax : 0.f;
                        // a row without a reference has nothing to rescale (and its
                        // first maximum may lie below -128: exp2(-dlt) = inf)
                        const float alpha = thr[m] == -INFINITY ? 0.f : fast_exp2(-dlt);
                        mref[m] = raise ? dlt - negm[m] : mref[m];
                        const bool seen = mref[m] != -INFINITY;
                        negm[m] = seen ? -mref[m] : 0.f;
                        negm4[m] = f32x4{negm[m], negm[m], negm[m], negm[m]};
                        thr[m] = seen ? kLazy : -INFINITY;
                        if (R > 1) refresh_addends(m);
                        if constexpr (kMfmaSum)
                            lsum[m] *= alpha;
                        else
                            lrow[m] *= alpha;
#pragma unroll
                        for (int db = 0; db < C::kDB; ++db) oacc[m][db] *= alpha;
#pragma unroll
                        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
                            for (int r = 0; r < 4; ++r) y[bi][r] -= dlt;
                    }
                    float p[2][4];
#pragma unroll
                    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
                        for (int r = 0; r < 4; ++r) p[bi][r] = fast_exp2(y[bi][r]);
                    pf[m] = x8{Tr<T>::cvt(p[0][0]), Tr<T>::cvt(p[0][1]), Tr<T>::cvt(p[0][2]),
                               Tr<T>::cvt(p[0][3]), Tr<T>::cvt(p[1][0]), Tr<T>::cvt(p[1][1]),
                               Tr<T>::cvt(p[1][2]), Tr<T>::cvt(p[1][3])};
                    if constexpr (!kMfmaSum) lrow[m] = row_sum8<T>(pf[m], p, lrow[m]);
                }

                // ---- O^T += V^T P^T (and the row sums, ones^T P^T) ----
                if (!kEarlyV) read_v();
#pragma unroll
                for (int db = 0; db < C::kDB; ++db)
#pragma unroll
                    for (int m = 0; m < QM; ++m) oacc[m][db] = Tr<T>::mma(vf[db], pf[m], oacc[m][db]);
                if constexpr (kMfmaSum) {
#pragma unroll
                    for (int m = 0; m < QM; ++m) lsum[m] = Tr<T>::mma(ones, pf[m], lsum[m]);
                }
            };
            // Tiles of two full blocks (kind 1, rows of more than two blocks) or
            // of two outer-full blocks (kind 2, short rows) are visited first, by
            // bodies without per-block branches, then (short rows) those with one
            // outer-full block; the order of tiles is free in the online softmax.
            run_tile_kinds<short_rows>(tiles, fullm, ofullm, tile);
            while (tiles) {
                const int tp = __builtin_ctzll(tiles) >> 1;
                tiles &= tiles - 1;
                tile(tp, std::integral_constant<int, 0>{});
            }
        }

        // the next stage's rows have landed, and this stage's buffer is free for
        // the loads issued next (no buffer is reused after the last stage)
        if (s + 1 < nst) {
            wait_vmem();
            __syncthreads();
        }
    }

    // ---- epilogue: normalise, store O (rounded once) and the natural-log LSE ----
#pragma unroll
    for (int m = 0; m < QM; ++m) {
        const float l = kMfmaSum ? lsum[m][0] : group_sum4(lrow[m]);
        if (!qvalid[m]) continue;
        const float inv = 1.f / l;
#pragma unroll
        for (int db = 0; db < C::kDB; ++db)
            st_x4<T>(og + qoff[m] + db * 16 + grp * 4, oacc[m][db] * inv);
        if (grp == 0) lseg[qoff[m] / D] = (mref[m] + __log2f(l)) * kLn2;
    }
}

// ---- host-side launch ----
// Largest number of 16-key blocks in any workgroup's halo (interior tiles).
static int max_halo_blocks(const Geo& g, int rank) {
    int nb = 1;
    for (int a = 0; a < rank; ++a) {
        const int n0 = group_len(g.L[a], g.d[a], 0);
        int e = std::min(g.T[a], n0) + g.k[a] - 1;
        e = std::min(e, n0);
        nb *= (a == rank - 1) ? (e + 15) / 16 : e;
    }
    return nb;
}

// Largest number of 16-key blocks in one halo row (interior tiles).
static int max_row_blocks(const Geo& g, int rank) {
    const int a = rank - 1;
    const int n0 = group_len(g.L[a], g.d[a], 0);
    const int e = std::min(std::min(g.T[a], n0) + g.k[a] - 1, n0);
    return (e + 15) / 16;
}

template <int R, int D, typename T, int QM, int SB, int W = 4>
static hipError_t launch_fwd_inst(const Geo& g, const void* q, const void* k, const void* v,
                                  void* o, float* lse, float scale, hipStream_t stream) {
    using C = FwdCfg<R, D, T, QM, SB, W>;
    // The register bound asks for no more workgroups per CU than a CU's
    // 160 KiB of LDS holds, with double buffers (stages of 16 blocks are used
    // only when the halo fits in one: single).
    static_assert(fwd_min_blocks<D, T, QM, W>() * (SB >= 16 ? 1 : 2) * C::kBufBytes <= 160 * 1024,
                  "register bound beyond the LDS occupancy");
    if (g.WGd[0] * g.WGd[1] * g.WGd[2] != W) return hipErrorInvalidConfiguration;
    const bool short_rows = R > 1 && max_row_blocks(g, R) <= 2;
    auto kern = na_fwd_kernel<R, D, T, QM, SB, 0, W>;
    if constexpr (R > 1)  // (1-D halos have one row: never short)
        if (short_rows) kern = na_fwd_kernel<R, D, T, QM, SB, 1, W>;
    const int nst_max = (max_halo_blocks(g, R) + SB - 1) / SB;
    const size_t lds = (nst_max > 1 ? 2 : 1) * C::kBufBytes;
    if (lds > 65536) {
        hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (e != hipSuccess) return e;
    }
    hipLaunchKernelGGL(kern, dim3(g.nwg), dim3(C::kThreads), lds, stream, g,
                       static_cast<const T*>(q), static_cast<const T*>(k),
                       static_cast<const T*>(v), static_cast<T*>(o), lse, scale * kLog2e);
    return hipGetLastError();
}

template <int R, int D, typename T>
static hipError_t launch_fwd_qm(const Geo& g, int qm, const void* q, const void* k, const void* v,
                                void* o, float* lse, float scale, hipStream_t stream) {
    if constexpr (sizeof(T) == 4) {
        if (qm == 1) return launch_fwd_inst<R, D, T, 1, 2>(g, q, k, v, o, lse, scale, stream);
        return launch_fwd_inst<R, D, T, 2, 2>(g, q, k, v, o, lse, scale, stream);
    } else {
        // One block per wave at D = 128: stages of half the keys, so that the
        // four waves per SIMD the registers allow also fit in LDS.
        constexpr int kSB1 = D == 128 ? 2 : 4;
        // 1-D: eight waves share each (twice as large) stage
        if constexpr (R == 1) {
            if (g.WGd[0] == 8) {
                if (qm == 1)
                    return launch_fwd_inst<R, D, T, 1, kSB1 * 2, 8>(g, q, k, v, o, lse, scale, stream);
                return launch_fwd_inst<R, D, T, 2, 8, 8>(g, q, k, v, o, lse, scale, stream);
            }
        }
        // one LDS stage covering the whole halo when it is small and D is 32
        if constexpr (D == 32) {
            if (max_halo_blocks(g, R) <= 16) {
                if (qm == 1) return launch_fwd_inst<R, D, T, 1, 16>(g, q, k, v, o, lse, scale, stream);
                return launch_fwd_inst<R, D, T, 2, 16>(g, q, k, v, o, lse, scale, stream);
            }
        }
        if (qm == 1) return launch_fwd_inst<R, D, T, 1, kSB1>(g, q, k, v, o, lse, scale, stream);
        return launch_fwd_inst<R, D, T, 2, 4>(g, q, k, v, o, lse, scale, stream);
    }
}

template <int R, typename T>
static hipError_t launch_fwd_d(const Geo& g, int D, int qm, const void* q, const void* k,
                               const void* v, void* o, float* lse, float scale, hipStream_t s) {
    switch (D) {
        case 32: return launch_fwd_qm<R, 32, T>(g, qm, q, k, v, o, lse, scale, s);
        case 64: return launch_fwd_qm<R, 64, T>(g, qm, q, k, v, o, lse, scale, s);
        case 128: return launch_fwd_qm<R, 128, T>(g, qm, q, k, v, o, lse, scale, s);
    }
    return hipErrorInvalidValue;
}

template <typename T>
static hipError_t launch_fwd_r(const Geo& g, int rank, int D, int qm, const void* q, const void* k,
                               const void* v, void* o, float* lse, float scale, hipStream_t s) {
    switch (rank) {
        case 1: return launch_fwd_d<1, T>(g, D, qm, q, k, v, o, lse, scale, s);
        case 2: return launch_fwd_d<2, T>(g, D, qm, q, k, v, o, lse, scale, s);
        case 3: return launch_fwd_d<3, T>(g, D, qm, q, k, v, o, lse, scale, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_forward(const Geo& g, int rank, int D, int dtype, int qm, const void* q,
                          const void* k, const void* v, void* o, float* lse, float scale,
                          hipStream_t s) {
    switch (dtype) {
        case 0: return launch_fwd_r<float>(g, rank, D, qm, q, k, v, o, lse, scale, s);
        case 1: return launch_fwd_r<_Float16>(g, rank, D, qm, q, k, v, o, lse, scale, s);
        case 2: return launch_fwd_r<__bf16>(g, rank, D, qm, q, k, v, o, lse, scale, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace na
