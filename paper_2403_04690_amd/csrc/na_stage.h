// na_stage.h -- direct global -> LDS staging of token rows, the swizzled LDS
// row layout the matrix-core fragments are read from, and the halo geometry
// those rows come from.
#pragma once

#include <type_traits>

#include "na_common.h"

namespace na {

// A box of tokens in group coordinates, [lo, lo + E) per axis, cut into rows
// along the innermost axis and each row into 16-token blocks (rows are padded
// to a multiple of 16; padding slots hold a stand-in token and are always
// masked).
template <int R>
struct Box {
    int lo[kMaxRank];
    int E[kMaxRank];
    int nbr;  // blocks per row
    int nb;   // total blocks
    FastDiv fd_nbr;
    FastDiv fd_E[kMaxRank];
    // token (within the (batch, head) slice) of the box's first position, and
    // the token distance of one step along each axis in group coordinates
    int tok_lo;
    int tstride[kMaxRank];

    // Block counts and divisors; gc[] is the dilation group of each axis.
    __device__ __forceinline__ void finish(const Geo& g, const int* gc) {
        nbr = (E[R - 1] + 15) >> 4;
        nb = nbr;
#pragma unroll
        for (int a = 0; a < R - 1; ++a) nb *= E[a];
        if constexpr (R > 1) fd_nbr.init(nbr);  // (1-D boxes are one row)
#pragma unroll
        for (int a = 1; a < R - 1; ++a) fd_E[a].init(E[a]);
        tok_lo = 0;
#pragma unroll
        for (int a = 0; a < R; ++a) {
            tstride[a] = g.d[a] * g.ts[a];
            tok_lo += (gc[a] + g.d[a] * lo[a]) * g.ts[a];
        }
    }

    // Outer coordinates (relative to lo) and first inner coordinate of block b
    // (blocks past the box get coordinates past it too).
    __device__ __forceinline__ void block_coords(int b, int* oc, int& inner0) const {
        if constexpr (R == 1) {  // one row: no division
            inner0 = b * 16;
            return;
        }
        int row = fd_nbr.div(b);
        inner0 = (b - row * nbr) * 16;
#pragma unroll
        for (int a = R - 2; a >= 1; --a) {
            const int nx = fd_E[a].div(row);
            oc[a] = row - nx * E[a];
            row = nx;
        }
        if (R >= 2) oc[0] = row;
    }

    // Token (within the (batch, head) slice) of slot 0 of block b, and how many
    // slots of the block hold a token of the box (0 for blocks past the end).
    // Slot j of the block is token + j * g.d[R-1].
    __device__ __forceinline__ int block_token(int b, int& valid) const {
        int oc[kMaxRank];
        int inner0;
        block_coords(b, oc, inner0);
        oc[R - 1] = inner0;
        const int left = E[R - 1] - inner0;
        valid = b < nb ? (left > 16 ? 16 : left) : 0;
        int tok = tok_lo;
#pragma unroll
        for (int a = 0; a < R; ++a) tok += oc[a] * tstride[a];
        return tok;
    }
};

// Per-wave block tests against a box of the other side: a block is relevant
// when it intersects [lo, hi) on every axis, and full when it lies inside
// [flo, fhi) on every axis (all its pairs with the wave's tokens are valid).
// Each range is kept as its start and its length (0 when empty), so that
// every test is one unsigned comparison.
template <int R>
struct WaveRange {
    int lo[kMaxRank], rlen[kMaxRank], flo[kMaxRank], flen[kMaxRank];
    int ilen;  // inner axis: blocks [i0, i0 + 16) meeting [lo, hi) have i0 - lo + 15 < ilen
    int iflen;  // inner axis: blocks inside [flo, fhi) have i0 - flo < iflen

    // Axis a: relevant range [lo_, hi_) (never empty), full range [flo_, fhi_).
    __device__ __forceinline__ void set(int a, int lo_, int hi_, int flo_, int fhi_) {
        lo[a] = lo_;
        rlen[a] = hi_ - lo_;
        flo[a] = flo_;
        flen[a] = fhi_ > flo_ ? fhi_ - flo_ : 0;
        if (a == R - 1) {
            ilen = hi_ - lo_ + 15;
            iflen = fhi_ - flo_ > 15 ? fhi_ - flo_ - 15 : 0;
        }
    }

    // rel: block b meets some window of the wave's queries; full: it lies
    // inside all of them; outer_full: inside all of them along the outer axes
    // (the innermost axis not tested).
    __device__ __forceinline__ void test(const Box<R>& box, int b, int* oc, int& inner0, bool& rel,
                                         bool& full, bool& outer_full) const {
        box.block_coords(b, oc, inner0);
        const bool in_box = b < box.nb;
        bool r_ = in_box, f_ = in_box;
#pragma unroll
        for (int a = 0; a < R - 1; ++a) {
            r_ = r_ & ((unsigned)(oc[a] - lo[a]) < (unsigned)rlen[a]);
            f_ = f_ & ((unsigned)(oc[a] - flo[a]) < (unsigned)flen[a]);
        }
        outer_full = f_;
        rel = r_ & ((unsigned)(inner0 - lo[R - 1] + 15) < (unsigned)ilen);
        full = f_ & ((unsigned)(inner0 - flo[R - 1]) < (unsigned)iflen);
    }
    __device__ __forceinline__ void test(const Box<R>& box, int b, int* oc, int& inner0, bool& rel,
                                         bool& full) const {
        bool outer_full;
        test(box, b, oc, inner0, rel, full, outer_full);
    }
};

// A wave's block tests taken 64 blocks at a time, one block per lane, instead
// of once per stage: a stage of SB blocks (SB divides 64) reads its bits from
// the chunk's masks, and a block's coordinates back from the lane that tested
// it.  Stages of 16 blocks or more (a whole halo, staged once) are tested
// stage by stage, with no chunk bookkeeping.
template <int R, int SB>
struct ChunkTests {
    static_assert(64 % SB == 0, "stages tile the 64-block chunks");
    static constexpr int kChunk = SB >= 16 ? SB : 64;  // blocks tested at a time
    static constexpr uint64_t kSel = SB == 64 ? ~0ull : (1ull << SB) - 1;
    int loc[kMaxRank], lin0;  // this lane's block: outer coordinates, first inner coordinate
    uint64_t rel, full, ofull;  // the chunk's blocks: relevant, full, full along the outer axes
    int j0;  // the stage's first block within the chunk

    // Stage s (stages are visited in order from 0).
    __device__ __forceinline__ void stage(const WaveRange<R>& wr, const Box<R>& box, int s,
                                          int lane) {
        j0 = (s * SB) & (kChunk - 1);
        if (j0 == 0) {
            bool r, f, o;
            wr.test(box, s * SB + lane, loc, lin0, r, f, o);
            rel = __builtin_amdgcn_ballot_w64(r);
            full = __builtin_amdgcn_ballot_w64(f);
            ofull = __builtin_amdgcn_ballot_w64(o);
        }
    }
    // bit j: block s * SB + j of the stage
    __device__ __forceinline__ uint64_t rel_bits() const { return (rel >> j0) & kSel; }
    __device__ __forceinline__ uint64_t full_bits() const { return (full >> j0) & kSel; }
    __device__ __forceinline__ uint64_t ofull_bits() const { return (ofull >> j0) & kSel; }
    // first inner coordinate and outer coordinate a of the stage's block j
    __device__ __forceinline__ int inner0(int j) const {
        return __builtin_amdgcn_readlane(lin0, j0 + j);
    }
    __device__ __forceinline__ int outer(int j, int a) const {
        return __builtin_amdgcn_readlane(loc[a], j0 + j);
    }
};

// Runs the tiles (bit 2 tp of `tiles`: block pair tp) whose kind allows a
// specialised body, removing them from `tiles`, which keeps the general ones
// (kind 0).  Kinds: 1 both blocks full (rows of more than two blocks); for
// short rows, 2 both blocks full along the outer axes, 3 / 4 only the first /
// second.  The order of tiles is free in the online softmax and in the sums.
template <bool SHORT_ROWS, typename F>
__device__ __forceinline__ void run_tile_kinds(uint64_t& tiles, uint64_t full, uint64_t ofull,
                                               F&& tile) {
    auto run = [&](uint64_t set, auto kind) {
        while (set) {
            const int tp = __builtin_ctzll(set) >> 1;
            set &= set - 1;
            tile(tp, kind);
        }
    };
    if constexpr (SHORT_ROWS) {
        const uint64_t of0 = ofull & 0x5555555555555555ull;
        const uint64_t of1 = (ofull >> 1) & 0x5555555555555555ull;
        run(tiles & of0 & of1, std::integral_constant<int, 2>{});
        run(tiles & of0 & ~of1, std::integral_constant<int, 3>{});
        run(tiles & ~of0 & of1, std::integral_constant<int, 4>{});
        tiles &= ~(of0 | of1);
    } else {
        const uint64_t pairs = full & (full >> 1) & 0x5555555555555555ull;
        run(tiles & pairs, std::integral_constant<int, 1>{});
        tiles &= ~pairs;
    }
}

// ---------------------------------------------------------------------------
// LDS rows: D elements of T per token, row-major and unpadded, cut into
// 16-byte segments; segment s of row r is stored at position s ^ swz(r).
// The swizzle is linear in the low four row bits and was chosen (by an
// exhaustive search over such functions) so that both fragment reads below
// are free of bank conflicts whether the LDS serves 128 or 256 bytes a cycle:
//   * 16-byte reads of one segment down 16 consecutive rows (MFMA operands
//     whose contraction runs along D);
//   * transposed 8-byte reads of 4 consecutive rows x 2 adjacent segments per
//     16 lanes (operands whose contraction runs along the tokens).
// ---------------------------------------------------------------------------
template <typename T, int D>
struct Rows {
    static constexpr int kSegs = D * (int)sizeof(T) / 16;  // segments per row
    static constexpr int kRowBytes = D * (int)sizeof(T);
    static constexpr int kVec = 16 / (int)sizeof(T);  // elements per segment
    static_assert(kSegs == 4 || kSegs == 8 || kSegs == 16 || kSegs == 32, "segments per row");

    __device__ __forceinline__ static int swz(int r) {
        constexpr int c0 = kSegs == 4 ? 0 : kSegs == 32 ? 1 : 2;
        constexpr int c1 = kSegs == 4 ? 2 : kSegs == 32 ? 2 : 4;
        constexpr int c2 = kSegs == 4 ? 3 : kSegs == 8 ? 3 : kSegs == 16 ? 9 : 4;
        constexpr int c3 = kSegs == 32 ? 8 : 1;
        return (-(r & 1) & c0) ^ (-((r >> 1) & 1) & c1) ^ (-((r >> 2) & 1) & c2) ^
               (-((r >> 3) & 1) & c3);
    }
    // byte offset of logical segment s of row r
    __device__ __forceinline__ static int off(int r, int s) {
        return r * kRowBytes + ((s ^ swz(r)) << 4);
    }
};

// Waits until this wave's outstanding vector memory operations (including
// direct-to-LDS loads) have completed.
__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

typedef __attribute__((address_space(3))) void lds_void;

// Stages ROWS token rows into an LDS tile with 16-byte direct-to-LDS loads
// (no register round trip): wave instruction t writes the tile's 16-byte
// positions [64 t, 64 t + 64), i.e. 64 / kSegs rows of one 16-row block, and
// lane l loads the segment that the swizzle puts at position 64 t + l.
// Tokens missing from the box are replaced by token 0 of the slice (finite
// data that the masks exclude).  Several tensors with the same rows share one
// set of per-lane source offsets.  With BLOCKWISE, when a block takes several
// instructions, wave w of the W takes the consecutive ones [w * kPerWave,
// (w + 1) * kPerWave), so that one block decode serves all of a block's
// instructions (2-D / 3-D boxes, whose decode has divisions); otherwise the
// waves take the instructions round-robin (measured faster for 1-D boxes).
template <typename T, int D, int ROWS, int W = 4, bool BLOCKWISE = false>
struct DirectRows {
    using L = Rows<T, D>;
    static constexpr int kRowsPerInstr = 64 / L::kSegs;
    static constexpr int kInstr = ROWS * L::kSegs / 64;  // wave instructions per tensor
    static constexpr int kPerWave = (kInstr + W - 1) / W;
    // wave instruction u of this wave
    __device__ __forceinline__ static int instr(int wave, int u) {
        return BLOCKWISE && kRowsPerInstr < 16 ? wave * kPerWave + u : wave + W * u;
    }
    static_assert(ROWS % 16 == 0 && kInstr >= 1, "whole blocks per stage");
    int src[kPerWave];  // element offset (within the slice) of this lane's segment

    // Rows of stage-local blocks b0, b0 + 1, ... of the box; tstep is the token
    // distance between consecutive slots of a block.
    template <int R>
    __device__ __forceinline__ void compute(const Box<R>& box, int b0, int tstep, int wave,
                                            int lane) {
#pragma unroll
        for (int u = 0; u < kPerWave; ++u) {
            const int t = instr(wave, u);
            src[u] = 0;
            if (t < kInstr) {
                const int row0 = t * kRowsPerInstr;  // first stage-local row (uniform)
                int valid;
                const int tok0 = box.block_token(b0 + (row0 >> 4), valid);
                const int j = (row0 & 15) + lane / L::kSegs;
                const int seg = (lane % L::kSegs) ^ L::swz(j);
                const int tok = j < valid ? tok0 + j * tstep : 0;
                src[u] = tok * D + seg * L::kVec;
            }
        }
    }

    __device__ __forceinline__ void issue(const T* base, unsigned char* tile, int wave) const {
#pragma unroll
        for (int u = 0; u < kPerWave; ++u) {
            const int t = instr(wave, u);
            if (t < kInstr)
                __builtin_amdgcn_global_load_lds(static_cast<const void*>(base + src[u]),
                                                 (lds_void*)(tile + t * 1024), 16, 0, 0);
        }
    }
};

// 16-byte and 8-byte LDS reads.
__device__ __forceinline__ i32x4 lds16(const unsigned char* p) {
    return *reinterpret_cast<const i32x4*>(p);
}

// Operand fragment of 16 rows x 32 contraction slots whose contraction runs
// along D (MFMA A/B layout: lane l holds row l % 16, slots 8 (l / 16) .. +7
// = elements st * 32 + 8 (l / 16) .. +7 of its row).  rowoff[] is from
// frag_offsets(); tile points at the first of the 16 rows.
template <typename T, int D>
struct RowFrag {
    using L = Rows<T, D>;
    static constexpr int kKS = D / 32;
    static constexpr int kN = sizeof(T) == 2 ? 1 : 2;  // 16-byte reads per fragment
    int off[kKS][kN];
    __device__ __forceinline__ void init(int lane) {
        const int r = lane & 15, g = lane >> 4;
#pragma unroll
        for (int st = 0; st < kKS; ++st)
#pragma unroll
            for (int n = 0; n < kN; ++n) off[st][n] = L::off(r, (st * 32 + g * 8) / L::kVec + n);
    }
    __device__ __forceinline__ typename Tr<T>::x8 read(const unsigned char* tile, int st) const {
        using x8 = typename Tr<T>::x8;
        if constexpr (sizeof(T) == 2) {
            return __builtin_bit_cast(x8, lds16(tile + off[st][0]));
        } else {
            const f32x4 a = __builtin_bit_cast(f32x4, lds16(tile + off[st][0]));
            const f32x4 b = __builtin_bit_cast(f32x4, lds16(tile + off[st][1]));
            return x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
        }
    }
};

// Transposed operand fragment: 16 columns d = db*16 + (l % 16) of D against
// 32 token slots, slot j of lane l holding token row
//   4 (l / 16) + j          (j < 4)   and   16 + 4 (l / 16) + j - 4   (j >= 4)
// of a 32-row tile -- the token order of a result tile of two 16-token
// blocks (result lane l holds rows 4 (l / 16) .. +3 of each block), so a
// probability or gradient tile feeds the next product without a shuffle.
// 16-bit types use the gfx950 transposed LDS read (each 16-lane group
// gathers 4 rows x 16 columns); fp32 reads the eight values one by one.
template <typename T, int D>
struct ColFrag {
    using L = Rows<T, D>;
    static constexpr int kDB = D / 16;
    int off[kDB];
    __device__ __forceinline__ void init(int lane) {
        const int g = lane >> 4, i = lane & 15;
        if constexpr (sizeof(T) == 2) {
            // lane 16g + 4s + q supplies row 4g + s, columns db*16 + 4q .. +3
            const int r = 4 * g + (i >> 2), q = i & 3;
#pragma unroll
            for (int db = 0; db < kDB; ++db)
                off[db] = L::off(r, (db * 16 + 4 * q) / L::kVec) + (q & 1) * 8;
        } else {
#pragma unroll
            for (int db = 0; db < kDB; ++db) off[db] = 0;
        }
    }
    __device__ __forceinline__ typename Tr<T>::x8 read(const unsigned char* tile, int db,
                                                       int lane) const {
        using x8 = typename Tr<T>::x8;
        if constexpr (sizeof(T) == 2) {
            typedef short s16x4 __attribute__((ext_vector_type(4)));
            typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
            const i32x2 a = __builtin_bit_cast(
                i32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(tile + off[db])));
            const i32x2 b = __builtin_bit_cast(
                i32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                           (lds_s16x4*)(tile + 16 * L::kRowBytes + off[db])));
            return __builtin_bit_cast(x8, i32x4{a[0], a[1], b[0], b[1]});
        } else {
            const int g = lane >> 4, d = db * 16 + (lane & 15);
            x8 v;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                const int r = (j < 4 ? 0 : 16) + 4 * g + (j & 3);
                v[j] = *reinterpret_cast<const float*>(tile + L::off(r, d / L::kVec) +
                                                       (d % L::kVec) * 4);
            }
            return v;
        }
    }
};

}  // namespace na
