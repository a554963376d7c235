// na_bwd.hip -- fused neighborhood-attention backward for gfx950.
//
// The backward pass is built from the three operators of Sec. 3.1, each run
// fused so that no attention weight reaches global memory:
//   PN  dP = dO V^T        (PN applied to the output gradient and V)
//   NN  dQ = scale dA K    over each query's neighbourhood
//   IN  dK = scale dA^T Q, dV = P^T dO  over each key's inverse neighbourhood
// with dA = P * (dP - Delta), Delta = rowsum(dO * O), and P recomputed from
// the logsumexp saved by the forward pass.  One launch, two workgroup roles,
// no atomics and no workspace, so the result is deterministic:
//   dK/dV role  one workgroup per key tile; its queries are the union of the
//               tile's inverse neighbourhoods (Sec. 3.1: the relation is not
//               symmetric and a key may be attended by up to k + floor(k/2)
//               queries per axis); Delta of every staged query is formed
//               while staging, from the O and dO rows
//   dQ role     one workgroup per query tile over its key halo, like the
//               forward pass; Delta of its own queries from their fragments
// The roles are independent, so they share the GPU instead of running as
// consecutive launches.
#include <algorithm>
#include <type_traits>

#include "na_launch.h"
#include "na_stage.h"

namespace na {

// ---------------------------------------------------------------------------
// dQ: query-major, over each query tile's key halo.
// ---------------------------------------------------------------------------
template <int R, int D, typename T, int QM, int SB>
struct DqCfg {
    static constexpr int kThreads = 4 * kWave;
    static constexpr int kKeys = SB * 16;
    static constexpr int kTileBytes = kKeys * Rows<T, D>::kRowBytes;
    static constexpr size_t kBufBytes = 2 * kTileBytes;  // K rows, then V rows
    static constexpr int kKS = D / 32;
    static constexpr int kDB = D / 16;
    using Ld = DirectRows<T, D, kKeys, 4, (R > 1)>;
};

// SHORT = 1: every halo row holds at most two 16-key blocks (rank >= 2), so
// the inner-axis mask is a per-lane constant (chosen on the host).
// braw: the workgroup's index among the dQ-role workgroups.
template <int R, int D, typename T, int QM, int SB, int SHORT>
__device__ __forceinline__ void dq_role(const Geo& g, int braw, unsigned char* smem_raw,
                                        const T* __restrict__ qg, const T* __restrict__ kg,
                                        const T* __restrict__ vg, const T* __restrict__ og,
                                        const T* __restrict__ dog, const float* __restrict__ lseg,
                                        T* __restrict__ dqg, float scale_log2, float scale) {
    using C = DqCfg<R, D, T, QM, SB>;
    using x8 = typename Tr<T>::x8;
    constexpr int kRowB = Rows<T, D>::kRowBytes;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = uniform((tid >> 6) & (C::kThreads / kWave - 1));  // (bounds the staging loops)
    const int col = lane & 15;
    const int grp = lane >> 4;

    const int bid = xcd_remap(braw, g.nwg);
    int bh, gc[kMaxRank], tc[kMaxRank], n[kMaxRank], to[kMaxRank];
    decode_workgroup<R>(g, bid, bh, gc, tc, n);

    Box<R> halo;
#pragma unroll
    for (int a = 0; a < R; ++a) {
        to[a] = tc[a] * g.T[a];
        if (to[a] >= n[a]) return;
        const int last = min(to[a] + g.T[a], n[a]) - 1;
        const bool ca = g.causal[a] != 0;
        halo.lo[a] = win_start(to[a], n[a], g.k[a], ca);
        halo.E[a] = win_last(last, n[a], g.k[a], ca) + 1 - halo.lo[a];
    }
    halo.finish(g, gc);

    const size_t slice = (size_t)bh * g.N * D;
    const T* kb = kg + slice;
    const T* vb = vg + slice;

    // The first stage is issued as soon as the halo is known, so that its
    // loads are in flight during the per-wave and per-lane set-up below.
    const int tstep = g.d[R - 1];
    typename C::Ld ld;
    auto issue_stage = [&](int s, int buf) {
        ld.compute(halo, s * SB, tstep, wave, lane);
        unsigned char* tile = smem_raw + buf * C::kBufBytes;
        ld.issue(kb, tile, wave);
        ld.issue(vb, tile + C::kTileBytes, wave);
    };
    issue_stage(0, 0);

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

    int qs[QM][kMaxRank];
    bool qvalid[QM];
    size_t qoff[QM];
    x8 qf[QM][C::kKS], gf[QM][C::kKS], of[QM][C::kKS];
    float lse2[QM], dlt[QM];
#pragma unroll
    for (int m = 0; m < QM; ++m) {
        int c[kMaxRank];
        unravel_pow2<R>(m * 16 + col, g.lgWT, c);
        bool ok = wave_live;
        int tok = 0;
#pragma unroll
        for (int a = 0; a < R; ++a) {
            int p = wo[a] + c[a];
            if (p >= n[a]) ok = false;
            p = min(p, n[a] - 1);
            qs[m][a] = mask_start(p, n[a], g.k[a], g.causal[a] != 0) - halo.lo[a];
            tok += (gc[a] + g.d[a] * p) * g.ts[a];
        }
        qvalid[m] = ok;
        qoff[m] = slice + (size_t)tok * D;
#pragma unroll
        // unconditional: qoff points at a real (clamped) query even for absent
        // slots, whose results are discarded
        for (int s = 0; s < C::kKS; ++s) {
            qf[m][s] = ld_x8<T>(qg + qoff[m] + s * 32 + grp * 8);
            gf[m][s] = ld_x8<T>(dog + qoff[m] + s * 32 + grp * 8);
            of[m][s] = ld_x8<T>(og + qoff[m] + s * 32 + grp * 8);
        }
        lse2[m] = lseg[qoff[m] / D] * kLog2e;
    }

    RowFrag<T, D> rfr;
    ColFrag<T, D> cfr;
    rfr.init(lane);
    cfr.init(lane);

    f32x4 dqacc[QM][C::kDB];
#pragma unroll
    for (int m = 0; m < QM; ++m)
#pragma unroll
        for (int db = 0; db < C::kDB; ++db) dqacc[m][db] = f32x4{0.f, 0.f, 0.f, 0.f};
    // Halo rows of at most two 16-key blocks: the inner-axis test of this
    // lane's 4 key slots is fixed, folded with -lse2 into per-slot addends.
    constexpr bool short_rows = SHORT != 0 && R > 1;
    // Score addends folded into the accumulators (not for D = 128 or bf16,
    // as in the forward)
    constexpr bool kFoldAdd = D <= 64 && !std::is_same_v<T, __bf16>;
    f32x4 ain[QM][2];
#pragma unroll
    for (int m = 0; m < QM; ++m)
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int ib = halo.nbr == 2 ? bi : 0;
                ain[m][bi][r] =
                    (unsigned)(ib * 16 + grp * 4 + r - qs[m][R - 1]) < (unsigned)g.k[R - 1]
                        ? -lse2[m]
                        : -INFINITY;
            }

    const int nst = (halo.nb + SB - 1) / SB;
    // Delta = dO . O of this lane's queries: 4 lanes hold a query's D slots
#pragma unroll
    for (int m = 0; m < QM; ++m) {
        float part = 0.f;
#pragma unroll
        for (int s = 0; s < C::kKS; ++s) part = dot8<T>(of[m][s], gf[m][s], part);
        dlt[m] = group_sum4(part);
    }
    wait_vmem();
    __syncthreads();
    // -lse2 in all four slots: the accumulator seed of full tiles (kFoldAdd)
    f32x4 nlse4[QM];
#pragma unroll
    for (int m = 0; m < QM; ++m) nlse4[m] = f32x4{-lse2[m], -lse2[m], -lse2[m], -lse2[m]};
    // kFoldAdd: Q scaled once by c = scale*log2(e) and rounded to T
    if constexpr (kFoldAdd)
#pragma unroll
    for (int m = 0; m < QM; ++m)
#pragma unroll
        for (int st = 0; st < C::kKS; ++st)
#pragma unroll
            for (int j = 0; j < 8; ++j) qf[m][st][j] = Tr<T>::cvt((float)qf[m][st][j] * scale_log2);

    ChunkTests<R, SB> ct;  // this wave's block tests, 64 blocks at a time
    for (int s = 0; s < nst; ++s) {
        if (s + 1 < nst) issue_stage(s + 1, (s + 1) & 1);
        const unsigned char* ks = smem_raw + (s & 1) * C::kBufBytes;
        const unsigned char* vs = ks + C::kTileBytes;

        if (wave_live) {
            // blocks are tested one per lane, 64 at a time; only tiles with a
            // relevant block are visited, their coordinates read back from the
            // lanes
            ct.stage(wr, halo, s, lane);
            const uint64_t relm = ct.rel_bits();
            const uint64_t fullm = ct.full_bits();
            const uint64_t ofullm = ct.ofull_bits();
            uint64_t tiles = (relm | (relm >> 1)) & 0x5555555555555555ull;
            // The body of one tile (block pair tp), by kind, as in the forward:
            // 0 general; 1 both blocks inside every window of the wave's queries;
            // 2 short rows, both blocks inside every window along the outer axes;
            // 3 / 4 short rows, only the first / second block so.
            auto tile = [&](int tp, auto tile_kind) {
                constexpr int kKind = decltype(tile_kind)::value;
                constexpr bool kFull = kKind == 1;
                // block bi inside every range along the outer axes
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

                // Y^T = c K Q^T + A (A: -lse2 on valid pairs, -inf on masked; with
                // kFoldAdd the accumulator starts at A and Q is prescaled by c) and
                // dP^T - Delta = V dO^T - Delta (the accumulator starts at -Delta)
                auto score_addend = [&](int m, int bi) {
                    f32x4 add;
                    if (!short_rows && full[bi]) {
                        add = f32x4{-lse2[m], -lse2[m], -lse2[m], -lse2[m]};
                    } else {
                        bool outer_ok = rel[bi];
                        if (!kOF[bi]) {
#pragma unroll
                            for (int a = 0; a < R - 1; ++a)
                                outer_ok = outer_ok &&
                                           (unsigned)(boc[bi][a] - qs[m][a]) < (unsigned)g.k[a];
                        }
                        // generic rows: slot r is valid when base + r lies in [0, lim)
                        const int base = bin0[bi] + grp * 4 - qs[m][R - 1];
                        const unsigned lim = outer_ok ? (unsigned)g.k[R - 1] : 0u;
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            add[r] = short_rows ? (outer_ok ? ain[m][bi][r] : -INFINITY)
                                     : (unsigned)(base + r) < lim ? -lse2[m] : -INFINITY;
                    }
                    return add;
                };
                f32x4 sacc[QM][2], pacc[QM][2];
#pragma unroll
                for (int bi = 0; bi < 2; ++bi) {
                    if (rel[bi]) {
                        const int boff = (tp * 2 + bi) * 16 * kRowB;
#pragma unroll
                        for (int st = 0; st < C::kKS; ++st) {
                            const x8 kf = rfr.read(ks + boff, st);
                            const x8 vf = rfr.read(vs + boff, st);
#pragma unroll
                            for (int m = 0; m < QM; ++m) {
                                if (st > 0)
                                    sacc[m][bi] = Tr<T>::mma(kf, qf[m][st], sacc[m][bi]);
                                else if (kFoldAdd && !short_rows && full[bi])
                                    sacc[m][bi] = Tr<T>::mma(kf, qf[m][0], nlse4[m]);  // in place
                                else if (kFoldAdd && short_rows && kOF[bi])
                                    sacc[m][bi] = Tr<T>::mma(kf, qf[m][0], ain[m][bi]);  // in place
                                else
                                    sacc[m][bi] = Tr<T>::mma(kf, qf[m][0],
                                                             kFoldAdd ? score_addend(m, bi)
                                                                      : f32x4{0.f, 0.f, 0.f, 0.f});
                                const f32x4 nd = f32x4{-dlt[m], -dlt[m], -dlt[m], -dlt[m]};
                                pacc[m][bi] = Tr<T>::mma(vf, gf[m][st], st == 0 ? nd : pacc[m][bi]);
                            }
                        }
                    } else {
#pragma unroll
                        for (int m = 0; m < QM; ++m) {
                            const float s0 = kFoldAdd ? -INFINITY : 0.f;
                            sacc[m][bi] = f32x4{s0, s0, s0, s0};
                            pacc[m][bi] = f32x4{0.f, 0.f, 0.f, 0.f};
                        }
                    }
                }

                // dA^T = P^T (dP^T - Delta), P = exp2(Y^T)
                x8 dsf[QM];
#pragma unroll
                for (int m = 0; m < QM; ++m) {
                    float ds[2][4];
#pragma unroll
                    for (int bi = 0; bi < 2; ++bi) {
                        f32x4 y = sacc[m][bi];
                        if constexpr (!kFoldAdd) {
                            const f32x4 add = score_addend(m, bi);
#pragma unroll
                            for (int r = 0; r < 4; ++r) y[r] = fmaf(y[r], scale_log2, add[r]);
                        }
#pragma unroll
                        for (int r = 0; r < 4; ++r) ds[bi][r] = fast_exp2(y[r]) * pacc[m][bi][r];
                    }
                    dsf[m] = x8{Tr<T>::cvt(ds[0][0]), Tr<T>::cvt(ds[0][1]), Tr<T>::cvt(ds[0][2]),
                                Tr<T>::cvt(ds[0][3]), Tr<T>::cvt(ds[1][0]), Tr<T>::cvt(ds[1][1]),
                                Tr<T>::cvt(ds[1][2]), Tr<T>::cvt(ds[1][3])};
                }

                // dQ^T += K^T dA^T (K^T read transposed from the K rows)
#pragma unroll
                for (int db = 0; db < C::kDB; ++db) {
                    const x8 kf = cfr.read(ks + tp * 32 * kRowB, db, lane);
#pragma unroll
                    for (int m = 0; m < QM; ++m) dqacc[m][db] = Tr<T>::mma(kf, dsf[m], dqacc[m][db]);
                }
            };
            // the specialised tiles first (the order of tiles does not matter)
            run_tile_kinds<short_rows>(tiles, fullm, ofullm, tile);
            while (tiles) {
                const int tp = __builtin_ctzll(tiles) >> 1;
                tiles &= tiles - 1;
                tile(tp, std::integral_constant<int, 0>{});
            }
        }

        if (s + 1 < nst) {  // (no buffer is reused after the last stage)
            wait_vmem();
            __syncthreads();
        }
    }

#pragma unroll
    for (int m = 0; m < QM; ++m) {
        if (!qvalid[m]) continue;
#pragma unroll
        for (int db = 0; db < C::kDB; ++db)
            st_x4<T>(dqg + qoff[m] + db * 16 + grp * 4, dqacc[m][db] * scale);
    }
}

// ---------------------------------------------------------------------------
// dK, dV: key-major, over the union of the key tile's inverse neighbourhoods.
// ---------------------------------------------------------------------------
// DIN: -Delta of every query comes from memory (written by a pre-pass), so
// neither O rows nor a Delta pass are needed.
template <int R, int D, typename T, int KM, int SB, bool DIN = false>
struct DkvCfg {
    static constexpr int kThreads = 4 * kWave;
    static constexpr int kRows = SB * 16;  // queries per stage
    static constexpr int kTileBytes = kRows * Rows<T, D>::kRowBytes;
    // Without DIN, one staged query per thread (the whole box in one stage):
    // each thread forms Delta of its query from its O row in registers, and
    // no O tile is staged.  Otherwise O rows are staged beside Q and dO.
    static constexpr bool kRegDelta = !DIN && kRows == kThreads;
    static constexpr int kTiles = (DIN || kRegDelta) ? 2 : 3;
    // Q rows, dO rows, [O rows,] then fp32 -lse2 and -Delta per query
    static constexpr size_t kFloatOff = (size_t)kTiles * kTileBytes;
    static constexpr size_t kBufBytes = kFloatOff + 2 * kRows * sizeof(float);
    static constexpr int kKS = D / 32;
    static constexpr int kDB = D / 16;
    using Ld = DirectRows<T, D, kRows, 4, (R > 1)>;
};

// SHORT = 1: every query-box row holds at most two 16-query blocks (rank >= 2).
// braw: the workgroup's index among the nwk dK/dV-role workgroups (nwk is
// g.nwg rounded up to a multiple of the 8 XCDs; the surplus ones exit).
// DIN: ndg holds -Delta of every query ([B * H * N] fp32, from the pre-pass).
template <int R, int D, typename T, int KM, int SB, int SHORT, bool DIN>
__device__ __forceinline__ void dkdv_role(const Geo& g, int braw, int nwk,
                                          unsigned char* smem_raw, const T* __restrict__ qg,
                                          const T* __restrict__ kg, const T* __restrict__ vg,
                                          const T* __restrict__ og, const T* __restrict__ dog,
                                          const float* __restrict__ lseg,
                                          const float* __restrict__ ndg, T* __restrict__ dkg,
                                          T* __restrict__ dvg, float scale_log2, float scale) {
    using C = DkvCfg<R, D, T, KM, SB, DIN>;
    using x8 = typename Tr<T>::x8;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = uniform((tid >> 6) & (C::kThreads / kWave - 1));  // (bounds the staging loops)
    const int col = lane & 15;  // key column of this lane
    const int grp = lane >> 4;

    const int bid = xcd_remap(braw, nwk);
    if (bid >= g.nwg) return;
    int bh, gc[kMaxRank], tc[kMaxRank], n[kMaxRank], to[kMaxRank];
    decode_workgroup<R>(g, bid, bh, gc, tc, n);

    // key tile [to, last] and the box of queries attending to it
    Box<R> ibox;
#pragma unroll
    for (int a = 0; a < R; ++a) {
        to[a] = tc[a] * g.T[a];
        if (to[a] >= n[a]) return;
        const int last = min(to[a] + g.T[a], n[a]) - 1;
        const bool ca = g.causal[a] != 0;
        ibox.lo[a] = inv_lo(to[a], n[a], g.k[a], ca);
        ibox.E[a] = inv_hi(last, n[a], g.k[a], ca) + 1 - ibox.lo[a];
    }
    ibox.finish(g, gc);

    const size_t slice = (size_t)bh * g.N * D;
    const T* qb = qg + slice;
    const T* gb = dog + slice;
    const T* ob = og + slice;
    const float* lb = lseg + (size_t)bh * g.N;
    const float* nb_ = DIN ? ndg + (size_t)bh * g.N : nullptr;

    const int tstep = g.d[R - 1];
    typename C::Ld ld;
    using L = Rows<T, D>;
    // the stage's per-query values as loaded (row tid of the stage), and
    // whether the row holds a query; combined only where they are stored
    float lse_raw = 0.f, ndl_raw = 0.f;
    bool row_ok = false;
    i32x4 orow[L::kSegs];  // kRegDelta: this thread's O row
    auto issue_stage = [&](int s, int buf) {
        ld.compute(ibox, s * SB, tstep, wave, lane);
        unsigned char* tile = smem_raw + buf * C::kBufBytes;
        ld.issue(qb, tile, wave);
        ld.issue(gb, tile + C::kTileBytes, wave);
        if constexpr (!DIN && !C::kRegDelta) ld.issue(ob, tile + 2 * C::kTileBytes, wave);
        // Every thread loads (threads past the stage's rows read a real token
        // too, whose values are never stored), with nothing computed from the
        // loaded values here: they are combined only in put_floats, so that
        // no wait for them (nor for the staging loads above) is needed before
        // the stage's tiles run.
        {
            int valid;
            const int tok0 = ibox.block_token(s * SB + (tid >> 4), valid);
            row_ok = (tid & 15) < valid;
            const int tk = row_ok ? tok0 + (tid & 15) * tstep : 0;  // token 0: safe stand-in
            lse_raw = lb[tk];
            if constexpr (DIN) ndl_raw = nb_[tk];  // already -Delta
            if constexpr (C::kRegDelta) {
#pragma unroll
                for (int sg = 0; sg < L::kSegs; ++sg)
                    orow[sg] = ld16<i32x4>(ob + (size_t)tk * D + sg * L::kVec);
            }
        }
    };
    // The first stage is issued as soon as the query box is known, so that
    // its loads are in flight during the per-wave and per-lane set-up below.
    issue_stage(0, 0);

    // this wave's key sub-box: the queries that attend to any / all of its keys
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
        wr.set(a, inv_lo(f, n[a], g.k[a], ca) - ibox.lo[a],
               inv_hi(l, n[a], g.k[a], ca) + 1 - ibox.lo[a],
               inv_lo(l, n[a], g.k[a], ca) - ibox.lo[a],
               inv_hi(f, n[a], g.k[a], ca) + 1 - ibox.lo[a]);
    }

    // per-lane keys: group coordinates, K and V fragments
    int kc[KM][kMaxRank];
    bool kvalid[KM];
    size_t koff[KM];
    x8 kf[KM][C::kKS], vf[KM][C::kKS];
#pragma unroll
    for (int m = 0; m < KM; ++m) {
        int c[kMaxRank];
        unravel_pow2<R>(m * 16 + col, g.lgWT, c);
        bool ok = wave_live;
        int tok = 0;
#pragma unroll
        for (int a = 0; a < R; ++a) {
            int p = wo[a] + c[a];
            if (p >= n[a]) ok = false;
            p = min(p, n[a] - 1);
            kc[m][a] = p;
            tok += (gc[a] + g.d[a] * p) * g.ts[a];
        }
        kvalid[m] = ok;
        koff[m] = slice + (size_t)tok * D;
#pragma unroll
        // unconditional: koff points at a real (clamped) key even for absent
        // slots, whose results are discarded
        for (int s = 0; s < C::kKS; ++s) {
            kf[m][s] = ld_x8<T>(kg + koff[m] + s * 32 + grp * 8);
            vf[m][s] = ld_x8<T>(vg + koff[m] + s * 32 + grp * 8);
        }
    }

    // A query q attends to this lane's key j exactly when q lies in j's
    // inverse range [inv_lo(j), inv_hi(j)] on every axis (contiguous, since
    // window starts are non-decreasing): per lane, relative to the query box.
    int ilo[KM][kMaxRank], ispan[KM][kMaxRank];
#pragma unroll
    for (int m = 0; m < KM; ++m)
#pragma unroll
        for (int a = 0; a < R; ++a) {
            const bool ca = g.causal[a] != 0;
            const int lo = inv_lo(kc[m][a], n[a], g.k[a], ca);
            ilo[m][a] = lo - ibox.lo[a];
            ispan[m][a] = inv_hi(kc[m][a], n[a], g.k[a], ca) - lo;
        }
    // Query-box rows of at most two 16-query blocks: the inner-axis test of
    // this lane's 4 query slots is fixed, folded into 0 / -inf addends.
    constexpr bool short_rows = SHORT != 0 && R > 1;
    // Score addends folded into the accumulators (not for D = 128 or bf16,
    // as in the forward)
    constexpr bool kFoldAdd = D <= 64 && !std::is_same_v<T, __bf16>;
    float ain[KM][2][4];
#pragma unroll
    for (int m = 0; m < KM; ++m)
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int ib = ibox.nbr == 2 ? bi : 0;
                ain[m][bi][r] = (unsigned)(ib * 16 + grp * 4 + r - ilo[m][R - 1]) <=
                                        (unsigned)ispan[m][R - 1]
                                    ? 0.f
                                    : -INFINITY;
            }

    auto floats = [&](int buf) {
        return reinterpret_cast<float*>(smem_raw + buf * C::kBufBytes + C::kFloatOff);
    };
    // 16-byte dot product in fp32
    auto dot16 = [&](i32x4 a, i32x4 b, float acc) {
        if constexpr (sizeof(T) == 2) {
            return dot8<T>(__builtin_bit_cast(x8, a), __builtin_bit_cast(x8, b), acc);
        } else {
            const f32x4 x = __builtin_bit_cast(f32x4, a), y = __builtin_bit_cast(f32x4, b);
            return fmaf(x[3], y[3], fmaf(x[2], y[2], fmaf(x[1], y[1], fmaf(x[0], y[0], acc))));
        }
    };
    // Delta = dO . O of the stage's staged queries (dO from its LDS rows; O
    // from its LDS rows with kThreads / kRows lanes per query reduced by lane
    // shuffles, or from the thread's registers); the float area holds -lse2
    // and -Delta per staged query
    auto delta_pass = [&](int buf) {
        const unsigned char* gt = smem_raw + buf * C::kBufBytes + C::kTileBytes;
        if constexpr (DIN) {
            (void)gt;
        } else if constexpr (C::kRegDelta) {
            float acc = 0.f;
#pragma unroll
            for (int sg = 0; sg < L::kSegs; ++sg) acc = dot16(lds16(gt + L::off(tid, sg)), orow[sg], acc);
            floats(buf)[C::kRows + tid] = -acc;  // staged negated: -Delta
        } else {
            constexpr int kP = C::kThreads / C::kRows;
            constexpr int kSpt = (L::kSegs + kP - 1) / kP;
            const unsigned char* ot = gt + C::kTileBytes;
            const int row = tid / kP, part = tid % kP;
            float acc = 0.f;
#pragma unroll
            for (int i = 0; i < kSpt; ++i) {
                const int seg = part * kSpt + i;
                if (seg < L::kSegs) {
                    const int o = L::off(row, seg);
                    acc = dot16(lds16(gt + o), lds16(ot + o), acc);
                }
            }
#pragma unroll
            for (int w = 1; w < kP; w <<= 1) acc += __shfl_xor(acc, w, kWave);
            if (part == 0) floats(buf)[C::kRows + row] = -acc;  // staged negated: -Delta
        }
    };
    RowFrag<T, D> rfr;
    ColFrag<T, D> cfr;
    rfr.init(lane);
    cfr.init(lane);
    constexpr int kRowB = Rows<T, D>::kRowBytes;

    f32x4 dkacc[KM][C::kDB], dvacc[KM][C::kDB];
#pragma unroll
    for (int m = 0; m < KM; ++m)
#pragma unroll
        for (int d = 0; d < C::kDB; ++d) {
            dkacc[m][d] = f32x4{0.f, 0.f, 0.f, 0.f};
            dvacc[m][d] = f32x4{0.f, 0.f, 0.f, 0.f};
        }

    const int nst = (ibox.nb + SB - 1) / SB;
    // the per-query floats of a stage: -lse2, and -Delta when it comes from memory
    auto put_floats = [&](int buf) {
        if (tid < C::kRows) {
            floats(buf)[tid] = row_ok ? -lse_raw * kLog2e : 0.f;  // staged negated: -lse2
            if constexpr (DIN) floats(buf)[C::kRows + tid] = row_ok ? ndl_raw : 0.f;
        }
    };
    put_floats(0);
    wait_vmem();
    __syncthreads();
    delta_pass(0);
    // kFoldAdd: K scaled once by c = scale*log2(e) and rounded to T
    if constexpr (kFoldAdd)
#pragma unroll
    for (int m = 0; m < KM; ++m)
#pragma unroll
        for (int st = 0; st < C::kKS; ++st)
#pragma unroll
            for (int j = 0; j < 8; ++j) kf[m][st][j] = Tr<T>::cvt((float)kf[m][st][j] * scale_log2);
    if constexpr (!DIN) __syncthreads();  // Delta of the first stage written

    ChunkTests<R, SB> ct;  // this wave's block tests, 64 blocks at a time
    for (int s = 0; s < nst; ++s) {
        if (s + 1 < nst) issue_stage(s + 1, (s + 1) & 1);
        const unsigned char* qs = smem_raw + (s & 1) * C::kBufBytes;
        const unsigned char* gs = qs + C::kTileBytes;
        const float* ls = floats(s & 1);
        const float* dls = ls + C::kRows;

        if (wave_live) {
            // blocks are tested one per lane, 64 at a time; only tiles with a
            // relevant block are visited, their coordinates read back from the
            // lanes
            ct.stage(wr, ibox, s, lane);
            const uint64_t relm = ct.rel_bits();
            const uint64_t fullm = ct.full_bits();
            const uint64_t ofullm = ct.ofull_bits();
            uint64_t tiles = (relm | (relm >> 1)) & 0x5555555555555555ull;
            // The body of one tile (block pair tp), by kind: 0 general; 1 both
            // query blocks attend every key of the wave; 2 short rows, both
            // blocks inside the wave's inverse ranges along the outer axes; 3 / 4
            // short rows, only the first / second block so.
            auto tile = [&](int tp, auto tile_kind) {
                constexpr int kKind = decltype(tile_kind)::value;
                constexpr bool kFull = kKind == 1;
                // block bi inside every range along the outer axes
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

                // -lse2 and -Delta of the 2 x 4 queries this lane holds
                f32x4 nlse[2], ndl[2];
#pragma unroll
                for (int bi = 0; bi < 2; ++bi) {
                    const int srow = (tp * 2 + bi) * 16 + grp * 4;
                    nlse[bi] = ld16<f32x4>(ls + srow);
                    ndl[bi] = ld16<f32x4>(dls + srow);
                }

                // Y = c Q K^T + A (A: -lse2 on valid pairs, -inf on masked; with
                // kFoldAdd the accumulator starts at A and K is prescaled by c) and
                // dP - Delta = dO V^T - Delta (rows: queries, columns: this wave's
                // keys; the accumulator starts at -Delta)
                auto score_addend = [&](int m, int bi) {
                    f32x4 add;
                    if (!short_rows && full[bi]) {
                        add = nlse[bi];
                    } else {
                        bool outer_ok = rel[bi];
                        if (!kOF[bi]) {
#pragma unroll
                            for (int a = 0; a < R - 1; ++a)
                                outer_ok = outer_ok && (unsigned)(boc[bi][a] - ilo[m][a]) <=
                                                           (unsigned)ispan[m][a];
                        }
                        // generic rows: slot r is valid when base + r lies in [0, lim)
                        const int base = bin0[bi] + grp * 4 - ilo[m][R - 1];
                        const unsigned lim = outer_ok ? (unsigned)ispan[m][R - 1] + 1u : 0u;
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            add[r] = short_rows ? (outer_ok ? nlse[bi][r] + ain[m][bi][r] : -INFINITY)
                                     : (unsigned)(base + r) < lim ? nlse[bi][r] : -INFINITY;
                    }
                    return add;
                };
                f32x4 sacc[KM][2], pacc[KM][2];
#pragma unroll
                for (int bi = 0; bi < 2; ++bi) {
                    if (rel[bi]) {
                        const int boff = (tp * 2 + bi) * 16 * kRowB;
#pragma unroll
                        for (int st = 0; st < C::kKS; ++st) {
                            const x8 qa = rfr.read(qs + boff, st);
                            const x8 ga = rfr.read(gs + boff, st);
#pragma unroll
                            for (int m = 0; m < KM; ++m) {
                                if (st > 0)
                                    sacc[m][bi] = Tr<T>::mma(qa, kf[m][st], sacc[m][bi]);
                                else if (kFoldAdd && !short_rows && full[bi])
                                    sacc[m][bi] = Tr<T>::mma(qa, kf[m][0], nlse[bi]);  // in place
                                else
                                    sacc[m][bi] = Tr<T>::mma(qa, kf[m][0],
                                                             kFoldAdd ? score_addend(m, bi)
                                                                      : f32x4{0.f, 0.f, 0.f, 0.f});
                                pacc[m][bi] = Tr<T>::mma(ga, vf[m][st], st == 0 ? ndl[bi] : pacc[m][bi]);
                            }
                        }
                    } else {
#pragma unroll
                        for (int m = 0; m < KM; ++m) {
                            const float s0 = kFoldAdd ? -INFINITY : 0.f;
                            sacc[m][bi] = f32x4{s0, s0, s0, s0};
                            pacc[m][bi] = f32x4{0.f, 0.f, 0.f, 0.f};
                        }
                    }
                }

                // P = exp2(Y), dA = P (dP - Delta)
                x8 pf[KM], dsf[KM];
#pragma unroll
                for (int m = 0; m < KM; ++m) {
                    float p[2][4], ds[2][4];
#pragma unroll
                    for (int bi = 0; bi < 2; ++bi) {
                        f32x4 y = sacc[m][bi];
                        if constexpr (!kFoldAdd) {
                            const f32x4 add = score_addend(m, bi);
#pragma unroll
                            for (int r = 0; r < 4; ++r) y[r] = fmaf(y[r], scale_log2, add[r]);
                        }
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const float pv = fast_exp2(y[r]);
                            p[bi][r] = pv;
                            ds[bi][r] = pv * pacc[m][bi][r];
                        }
                    }
                    pf[m] = x8{Tr<T>::cvt(p[0][0]), Tr<T>::cvt(p[0][1]), Tr<T>::cvt(p[0][2]),
                               Tr<T>::cvt(p[0][3]), Tr<T>::cvt(p[1][0]), Tr<T>::cvt(p[1][1]),
                               Tr<T>::cvt(p[1][2]), Tr<T>::cvt(p[1][3])};
                    dsf[m] = x8{Tr<T>::cvt(ds[0][0]), Tr<T>::cvt(ds[0][1]), Tr<T>::cvt(ds[0][2]),
                                Tr<T>::cvt(ds[0][3]), Tr<T>::cvt(ds[1][0]), Tr<T>::cvt(ds[1][1]),
                                Tr<T>::cvt(ds[1][2]), Tr<T>::cvt(ds[1][3])};
                }

                // dV^T += dO^T P and dK^T += Q^T dA (transposed reads of the rows)
#pragma unroll
                for (int d = 0; d < C::kDB; ++d) {
                    const x8 ga = cfr.read(gs + tp * 32 * kRowB, d, lane);
                    const x8 qa = cfr.read(qs + tp * 32 * kRowB, d, lane);
#pragma unroll
                    for (int m = 0; m < KM; ++m) {
                        dvacc[m][d] = Tr<T>::mma(ga, pf[m], dvacc[m][d]);
                        dkacc[m][d] = Tr<T>::mma(qa, dsf[m], dkacc[m][d]);
                    }
                }
                        };
            // the specialised tiles first (the order of tiles does not matter);
            // 16-bit types at D <= 64 only (the compiler fails on the others)
            if constexpr (sizeof(T) == 2 && D <= 64)
                run_tile_kinds<short_rows>(tiles, fullm, ofullm, tile);
            while (tiles) {
                const int tp = __builtin_ctzll(tiles) >> 1;
                tiles &= tiles - 1;
                tile(tp, std::integral_constant<int, 0>{});
            }
        }

        if (s + 1 < nst) {  // (no buffer is reused after the last stage)
            put_floats((s + 1) & 1);
            wait_vmem();
            __syncthreads();
            if (!DIN) {
                delta_pass((s + 1) & 1);
                __syncthreads();
            }
        }
    }

#pragma unroll
    for (int m = 0; m < KM; ++m) {
        if (!kvalid[m]) continue;
#pragma unroll
        for (int d = 0; d < C::kDB; ++d) {
            st_x4<T>(dkg + koff[m] + d * 16 + grp * 4, dkacc[m][d] * scale);
            st_x4<T>(dvg + koff[m] + d * 16 + grp * 4, dvacc[m][d]);
        }
    }
}

// ---------------------------------------------------------------------------
// the kernel: workgroups [0, nwk) take the dK/dV role, the next g.nwg the dQ
// role (dK/dV first: its workgroups carry more work and start earlier)
// ---------------------------------------------------------------------------
// 16-bit types with D <= 64 are held to 2 waves per SIMD (<= 256 registers),
// and to 3 (<= 168) for rank 1: there the few values that no longer fit are
// spilled outside the tile loop (the dQ role's per-stage state), and the
// third wave hides more of the tile loop's latency (1-D k = 1023 backward:
// -7 %).  Ranks 2 and 3 would spill inside the loop.
// ROLE 0 runs both roles in one grid; ROLE 1 only the dK/dV role (nwk
// workgroups) and ROLE 2 only the dQ role (g.nwg workgroups), each as a
// launch of its own with its own register budget.  ROLE 1 stages 128
// queries per stage at D = 64, double-buffered: about 67 KiB
// of LDS, so two workgroups share a CU, two waves per SIMD whatever the
// registers, and a tighter bound would only spill.  Rank 1 at D = 64 stages
// 64 queries instead (about 34 KiB), which leaves room for the third wave,
// and D = 32 stages 128 (about 34 KiB): four waves at rank 1, three above.
template <int R, int D, typename T, int QM, int ROLE>
constexpr int bwd_min_waves() {
    if constexpr (ROLE == 2) return sizeof(T) == 2 && D <= 64 ? (QM == 1 ? 5 : 3) : 2;
    if constexpr (ROLE == 1) return R == 1 && D == 64 ? 3 : (D == 32 ? (R == 1 ? 4 : 3) : 2);
    return sizeof(T) == 2 && D <= 64 ? (R == 1 ? 3 : 2) : 1;
}

template <int R, int D, typename T, int QM, int KM, int SBQ, int SBK, int SHORT, int ROLE>
__global__ __launch_bounds__(256, (bwd_min_waves<R, D, T, QM, ROLE>())) void na_bwd_kernel(Geo g, int nwk, const T* __restrict__ q,
                                                     const T* __restrict__ k,
                                                     const T* __restrict__ v,
                                                     const T* __restrict__ o,
                                                     const T* __restrict__ dout,
                                                     const float* __restrict__ lse,
                                                     const float* __restrict__ ndelta,
                                                     T* __restrict__ dq, T* __restrict__ dk,
                                                     T* __restrict__ dv, float scale_log2,
                                                     float scale) {
    extern __shared__ __align__(16) unsigned char smem_raw[];
    const int b = blockIdx.x;
    if constexpr (ROLE == 1) {
        dkdv_role<R, D, T, KM, SBK, SHORT, true>(g, b, nwk, smem_raw, q, k, v, o, dout, lse,
                                                 ndelta, dk, dv, scale_log2, scale);
    } else if constexpr (ROLE == 2) {
        dq_role<R, D, T, QM, SBQ, SHORT>(g, b, smem_raw, q, k, v, o, dout, lse, dq, scale_log2,
                                         scale);
    } else {
        if (b < nwk)
            dkdv_role<R, D, T, KM, SBK, SHORT, false>(g, b, nwk, smem_raw, q, k, v, o, dout, lse,
                                                      nullptr, dk, dv, scale_log2, scale);
        else
            dq_role<R, D, T, QM, SBQ, SHORT>(g, b - nwk, smem_raw, q, k, v, o, dout, lse, dq,
                                             scale_log2, scale);
    }
}

// ---------------------------------------------------------------------------
// host-side launch
// ---------------------------------------------------------------------------
// Longest extent along one axis, over every tile and both group lengths of a
// dilated axis, of a workgroup's key halo (inverse = false) or of the box of
// queries attending to its key tile (inverse = true).  Window starts grow by
// at most one per position, so a halo never exceeds min(T, n) + k - 1; an
// inverse box can (every key within k - 1 of the start is attended by query
// 0), so the tiles near a border are evaluated one by one and a single
// interior tile (extent T + k - 1) stands for the rest.  Causal axes have no
// such border growth.
static int max_box_extent(int L, int d, int k, int T, bool causal, bool inverse) {
    int best = 0;
    const int n0 = group_len(L, d, 0);
    for (int n = n0; n >= n0 - 1; --n) {
        if (n < n0 && L % d == 0) break;  // every group has length n0
        // along a causal axis both boxes are [start(first), last] and
        // [first, min(last + k - 1, n - 1)]: never wider than T + k - 1
        if (!inverse || causal) {
            best = std::max(best, std::min(std::min(T, n) + k - 1, n));
            continue;
        }
        const int nt = (n + T - 1) / T;
        const int edge = k / T + 2;  // tiles that can reach within k of a border
        for (int i = 0; i < nt; ++i) {
            if (i > edge && i < nt - edge) continue;
            const int to = i * T, last = std::min(to + T, n) - 1;
            best = std::max(best, inv_hi(last, n, k, false) + 1 - inv_lo(to, n, k, false));
        }
    }
    return best;
}

// 16-token blocks of the largest box with per-axis extents e[]: rows along
// the innermost axis are cut into blocks.
static int box_blocks(const int* e, int rank) {
    int nb = (e[rank - 1] + 15) / 16;
    for (int a = 0; a < rank - 1; ++a) nb *= e[a];
    return nb;
}

// Delta pre-pass of the split backward: nd[row] = -sum_c dO[row, c] O[row, c]
// in fp32, the lanes of a 16-byte segment group sharing a row.
template <typename T, int D>
__global__ __launch_bounds__(256) void na_delta_kernel(const T* __restrict__ o,
                                                       const T* __restrict__ dout,
                                                       float* __restrict__ nd, int64_t rows) {
    using L = Rows<T, D>;
    constexpr int kSegs = L::kSegs;  // lanes per row (a power of two dividing 64)
    const int seg = threadIdx.x % kSegs;
    const int64_t step = (int64_t)gridDim.x * (256 / kSegs);
    for (int64_t row = (int64_t)blockIdx.x * (256 / kSegs) + threadIdx.x / kSegs; row < rows;
         row += step) {
        const i32x4 a = ld16<i32x4>(o + row * D + seg * L::kVec);
        const i32x4 b = ld16<i32x4>(dout + row * D + seg * L::kVec);
        float acc;
        if constexpr (sizeof(T) == 2) {
            using x8 = typename Tr<T>::x8;
            acc = dot8<T>(__builtin_bit_cast(x8, a), __builtin_bit_cast(x8, b), 0.f);
        } else {
            const f32x4 x = __builtin_bit_cast(f32x4, a), y = __builtin_bit_cast(f32x4, b);
            acc = fmaf(x[3], y[3], fmaf(x[2], y[2], fmaf(x[1], y[1], x[0] * y[0])));
        }
#pragma unroll
        for (int w = 1; w < kSegs; w <<= 1) acc += __shfl_xor(acc, w, kWave);
        if (seg == 0) nd[row] = -acc;
    }
}

// hq / hk: most blocks in any dQ halo / dK-dV query box; a role whose boxes
// all fit in one stage gets a single LDS buffer.
//
// One launch runs both roles (dK/dV workgroups first).  The split form, for
// large 16-bit problems at D <= 64, runs three launches instead: a Delta
// pre-pass writing -Delta of every query into dq (scratch until the last
// launch overwrites it), the dK/dV role reading it (no O rows, no Delta pass,
// one barrier per stage, stages of SBS blocks), then the dQ role; each role
// runs at the occupancy its own registers and LDS allow.
template <int R, int D, typename T, int QM, int KM, int SBQ, int SBK>
static hipError_t launch_bwd_sb(const Geo& g, bool short_rows, bool split, int hq, int hk,
                                const void* q, const void* k, const void* v, const void* o,
                                const float* lse, const void* dout, void* dq, void* dk, void* dv,
                                float scale, hipStream_t stream) {
    const size_t lds_q = (hq > SBQ ? 2 : 1) * DqCfg<R, D, T, QM, SBQ>::kBufBytes;
    const size_t lds_k = (hk > SBK ? 2 : 1) * DkvCfg<R, D, T, KM, SBK>::kBufBytes;
    // No register bound asks for more waves per SIMD (workgroups of four
    // waves per CU) than a CU's 160 KiB of LDS holds, with double buffers
    // (stages of 16 blocks are used only when every box fits in one: single).
    constexpr size_t kCuLds = 160 * 1024;
    constexpr size_t kLdsQ = (SBQ >= 16 ? 1 : 2) * DqCfg<R, D, T, QM, SBQ>::kBufBytes;
    constexpr size_t kLdsK = (SBK >= 16 ? 1 : 2) * DkvCfg<R, D, T, KM, SBK>::kBufBytes;
    static_assert(bwd_min_waves<R, D, T, QM, 0>() * (kLdsQ > kLdsK ? kLdsQ : kLdsK) <= kCuLds,
                  "one-launch register bound beyond the LDS occupancy");
    static_assert(bwd_min_waves<R, D, T, QM, 2>() * kLdsQ <= kCuLds,
                  "dQ-launch register bound beyond the LDS occupancy");
    const int nwk = (g.nwg + 7) & ~7;
    auto launch = [&](auto kern, size_t lds, int grid, const float* nd) -> hipError_t {
        if (lds > 65536) {
            hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                               (int)lds);
            if (e != hipSuccess) return e;
        }
        hipLaunchKernelGGL(kern, dim3((unsigned)grid), dim3(4 * kWave), lds, stream, g, nwk,
                           static_cast<const T*>(q), static_cast<const T*>(k),
                           static_cast<const T*>(v), static_cast<const T*>(o),
                           static_cast<const T*>(dout), lse, nd, static_cast<T*>(dq),
                           static_cast<T*>(dk), static_cast<T*>(dv), scale * kLog2e, scale);
        return hipGetLastError();
    };
    if constexpr (sizeof(T) == 2 && D <= 64) {
        if (split) {
            // query blocks per stage of the dK/dV launch (see bwd_min_waves)
            constexpr int SBS = D == 32 ? 8 : (R == 1 ? 4 : 8);
            const size_t lds_ks = (hk > SBS ? 2 : 1) * DkvCfg<R, D, T, KM, SBS, true>::kBufBytes;
            static_assert(bwd_min_waves<R, D, T, QM, 1>() * 2 *
                                  DkvCfg<R, D, T, KM, SBS, true>::kBufBytes <= kCuLds,
                          "dK/dV-launch register bound beyond the LDS occupancy");
            auto kk = na_bwd_kernel<R, D, T, QM, KM, SBQ, SBS, 0, 1>;
            auto kq = na_bwd_kernel<R, D, T, QM, KM, SBQ, SBK, 0, 2>;
            if constexpr (R > 1)
                if (short_rows) {
                    kk = na_bwd_kernel<R, D, T, QM, KM, SBQ, SBS, 1, 1>;
                    kq = na_bwd_kernel<R, D, T, QM, KM, SBQ, SBK, 1, 2>;
                }
            float* nd = static_cast<float*>(dq);
            const int64_t rows = (int64_t)g.BH * g.N;
            constexpr int kRowsPerBlock = 256 / Rows<T, D>::kSegs;
            const int64_t blocks = std::min<int64_t>((rows + kRowsPerBlock - 1) / kRowsPerBlock,
                                                     int64_t(1) << 18);
            hipLaunchKernelGGL((na_delta_kernel<T, D>), dim3((unsigned)blocks), dim3(256), 0,
                               stream, static_cast<const T*>(o), static_cast<const T*>(dout), nd,
                               rows);
            hipError_t e = hipGetLastError();
            if (e != hipSuccess) return e;
            e = launch(kk, lds_ks, nwk, nd);
            if (e != hipSuccess) return e;
            return launch(kq, lds_q, g.nwg, nullptr);
        }
    }
    (void)split;
    auto kern = na_bwd_kernel<R, D, T, QM, KM, SBQ, SBK, 0, 0>;
    if constexpr (R > 1)  // (1-D boxes have one row: never short)
        if (short_rows) kern = na_bwd_kernel<R, D, T, QM, KM, SBQ, SBK, 1, 0>;
    return launch(kern, std::max(lds_q, lds_k), nwk + g.nwg, nullptr);
}

template <int R, int D, typename T, int QM, int KM>
static hipError_t launch_bwd_inst(const Geo& g, const void* q, const void* k, const void* v,
                                  const void* o, const float* lse, const void* dout, void* dq,
                                  void* dk, void* dv, float scale, hipStream_t stream) {
    int eq[kMaxRank], ek[kMaxRank];
    for (int a = 0; a < R; ++a) {
        eq[a] = max_box_extent(g.L[a], g.d[a], g.k[a], g.T[a], g.causal[a] != 0, false);
        ek[a] = max_box_extent(g.L[a], g.d[a], g.k[a], g.T[a], g.causal[a] != 0, true);
    }
    const int hq = box_blocks(eq, R), hk = box_blocks(ek, R);
    // rows of every halo (dQ) and query box (dK/dV) hold at most 2 blocks
    const bool short_rows = R > 1 && (eq[R - 1] + 15) / 16 <= 2 && (ek[R - 1] + 15) / 16 <= 2;
    const bool split = g.bwd_split != 0;  // chosen on the host with the tiling
    // D = 32, 16-bit: boxes of up to 16 blocks are staged whole (one stage)
    if constexpr (sizeof(T) == 2 && D == 32) {
        if (hq <= 16 && hk <= 16)
            return launch_bwd_sb<R, D, T, QM, KM, 16, 16>(g, short_rows, split, hq, hk, q, k, v,
                                                          o, lse, dout, dq, dk, dv, scale, stream);
    }
    constexpr int SBQ = sizeof(T) == 4 ? 2 : 4;
    constexpr int SBK = (sizeof(T) == 4 || D == 128) ? 2 : 4;
    return launch_bwd_sb<R, D, T, QM, KM, SBQ, SBK>(g, short_rows, split, hq, hk, q, k, v, o, lse,
                                                    dout, dq, dk, dv, scale, stream);
}

template <int R, int D, typename T>
static hipError_t launch_bwd_m(const Geo& g, int m, const void* q, const void* k, const void* v,
                               const void* o, const float* lse, const void* dout, void* dq,
                               void* dk, void* dv, float scale, hipStream_t s) {
    if (m == 1) return launch_bwd_inst<R, D, T, 1, 1>(g, q, k, v, o, lse, dout, dq, dk, dv, scale, s);
    return launch_bwd_inst<R, D, T, 2, 2>(g, q, k, v, o, lse, dout, dq, dk, dv, scale, s);
}

template <int R, typename T>
static hipError_t launch_bwd_d(const Geo& g, int D, int m, const void* q, const void* k,
                               const void* v, const void* o, const float* lse, const void* dout,
                               void* dq, void* dk, void* dv, float scale, hipStream_t s) {
    switch (D) {
        case 32: return launch_bwd_m<R, 32, T>(g, m, q, k, v, o, lse, dout, dq, dk, dv, scale, s);
        case 64: return launch_bwd_m<R, 64, T>(g, m, q, k, v, o, lse, dout, dq, dk, dv, scale, s);
        case 128: return launch_bwd_m<R, 128, T>(g, m, q, k, v, o, lse, dout, dq, dk, dv, scale, s);
    }
    return hipErrorInvalidValue;
}

template <typename T>
static hipError_t launch_bwd_r(const Geo& g, int rank, int D, int m, const void* q, const void* k,
                               const void* v, const void* o, const float* lse, const void* dout,
                               void* dq, void* dk, void* dv, float scale, hipStream_t s) {
    switch (rank) {
        case 1: return launch_bwd_d<1, T>(g, D, m, q, k, v, o, lse, dout, dq, dk, dv, scale, s);
        case 2: return launch_bwd_d<2, T>(g, D, m, q, k, v, o, lse, dout, dq, dk, dv, scale, s);
        case 3: return launch_bwd_d<3, T>(g, D, m, q, k, v, o, lse, dout, dq, dk, dv, scale, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_backward(const Geo& g, int rank, int D, int dtype, int m, const void* q,
                           const void* k, const void* v, const void* o, const float* lse,
                           const void* dout, void* dq, void* dk, void* dv, float scale,
                           hipStream_t s) {
    switch (dtype) {
        case 0: return launch_bwd_r<float>(g, rank, D, m, q, k, v, o, lse, dout, dq, dk, dv, scale, s);
        case 1: return launch_bwd_r<_Float16>(g, rank, D, m, q, k, v, o, lse, dout, dq, dk, dv, scale, s);
        case 2: return launch_bwd_r<__bf16>(g, rank, D, m, q, k, v, o, lse, dout, dq, dk, dv, scale, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace na
