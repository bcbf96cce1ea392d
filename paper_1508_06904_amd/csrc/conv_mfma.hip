// Convolution over the fragment batch as an MFMA implicit GEMM (gfx950).
//
// Every fragment is an independent signal (Definition "fragmentwise
// evaluation", Sect. 4.2), so all fragments of a layer form one batch of
// ordinary valid convolutions (Sect. 3.3 and its 2-D form in Sect. 6.1):
//   out[f][y][x][o] = act( bias[o] + sum_{t_h,t_w,i} W[o][i][t_h][t_w] * in[f][y+t_h][x+t_w][i] )
// As a GEMM: M = output samples (a TH x TW spatial tile of one fragment per
// workgroup), N = output channels, K = fh * fw * Cin.
//
// Workgroup = 4 wavefronts of 64 lanes; each wave owns a (32*MT) x (32*NT) block
// of the output tile (128 x 64 for the wide layers: the wider the wave tile, the
// fewer operand bytes per flop), computed with 32x32 MFMA tiles:
//   binary32:  v_mfma_f32_32x32x2_f32   (K = 2 per issue)
//   bfloat16:  v_mfma_f32_32x32x16_bf16 (K = 16 per issue), binary32 accumulation
// K loop: input channels in chunks of 64 bytes per sample (16 binary32 or 32
// bfloat16 channels) x filter taps; a step is one (chunk, tap) pair.  For each
// chunk the input halo tile (TH + fh - 1) x (TW + fw - 1) x chunk is staged in
// LDS once and read by all fh * fw taps (A operands; double-buffered across
// chunks when two workgroups still fit a CU).  The weights of a step, BN x
// chunk, go from global memory (L2-resident: every workgroup of an N block reads
// the same slices) straight into each lane's B registers two steps ahead: no
// LDS copy, one barrier per chunk.  Halo samples use an 80-byte LDS pitch so
// that the 32-byte operand reads of a wavefront spread over all banks.
//
// Spatial tiles may read a virtual zero border of pad_h x pad_w samples around
// every fragment (the input gradient of the backward pass); small fragments can
// instead be read as one flat sequence, and the dilated fashion tiles one signal
// by phase (see the kernel's parameters).
//
// K-index assignment inside one MFMA issue: lane half h (lanes 32h..32h+31)
// holds input channels h*8 + s (binary32, issue s of 8) or h*16 + 8s .. +7
// (bfloat16, issue s of 2) of the chunk; A and B use the same assignment, so
// every product pairs an input sample with its own weight.  The bfloat16
// variant with a folded 1x1 projection computes the transposed blocks
// (B^T A^T), which puts one sample and runs of four channels in each lane for
// its dot products.
//
// Epilogue: + bias, activation, masked store (edge tiles, padded channels) in
// the channels-last output layout, transposed through LDS into 16-byte stores
// (4 binary32 or 8 bfloat16 channels, round to nearest even, of one position).
#include <algorithm>

#include <type_traits>

#include "dev_common.h"
#include "dss_internal.h"

namespace dss {

typedef float floatx16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));   // one 16-byte unit

constexpr int kPitchBytes = 80;     // LDS bytes per staged sample / weight row
constexpr int kSlotsPerRow = kPitchBytes / 16;
constexpr int kChunkBytes = 64;     // bytes of one channel chunk per sample
constexpr int kMaxLds = 78 * 1024;  // two workgroups per CU (160 KB of LDS)
constexpr int kXcds = 8;            // accelerator complex dies of an MI355X
constexpr int kGroup = 16;          // neighbouring tiles scheduled together
constexpr int kSliceBlock = 2048;   // bytes of 32 weight rows x one 64-byte channel chunk

template <bool BF16, int WGM, int WGN, int MT, int NT>
struct MfmaCfg {
    static constexpr int ES = BF16 ? 2 : 4;
    static constexpr int CC = kChunkBytes / ES;        // channels per chunk
    static constexpr int BM = 32 * MT * WGM;            // output samples per workgroup
    static constexpr int BN = 32 * NT * WGN;            // output channels per workgroup
    static constexpr int THREADS = 64 * WGM * WGN;
};

// 16 zero bytes: the source of every staged unit that lies outside the fragment
// or in the zero-padded channels of the last chunk.
__device__ __attribute__((aligned(16))) const unsigned int g_zero16[4] = {0u, 0u, 0u, 0u};

__device__ __forceinline__ bf16x8 as_bf16x8(u32x4 v) { return __builtin_bit_cast(bf16x8, v); }

typedef __attribute__((address_space(3))) void lds_void;

// Direct global -> LDS copy of one 16-byte unit per active lane: the unit lands in
// LDS at wave_dst + 16 * lane (gfx950 global_load_lds_dwordx4).
__device__ __forceinline__ void dma16(const void* src, char* wave_dst) {
    __builtin_amdgcn_global_load_lds(src, (lds_void*)wave_dst, 16, 0, 0);
}

// Epilogue variants: kEpiStore writes the activations, kEpiProj the partial
// projections of a folded 1x1 convolution, kEpiPool the sliding-window maxima of
// a 1-D pool written straight to their fragments.
constexpr int kEpiStore = 0, kEpiProj = 1, kEpiPool = 2;

template <bool BF16, typename Tout, int WGM, int WGN, int MT, int NT, int EPI = kEpiStore>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void conv_mfma_kernel(
    const char* __restrict__ in,       // [F][Hin][Win][Cin] of BF16 ? bfloat16 : binary32
    int Hin, int Win, int Cin,
    const char* __restrict__ wp,       // packed [nb][chunk][th][tw][BN][chunk channels] (bfloat16: slices in lane order)
    const float* __restrict__ bias,    // [Cout_pad]
    int fh, int fw, int Cout, int act, int nchunks,
    Tout* __restrict__ out,            // [F][Hout][Wout][Cout]; kEpiPool: the fragments [k F][1][pool_U][Cout]
                                       // (unused with kEpiProj)
    int Hout, int Wout, int TH, int TW, int tilesY, int tilesX, int nbs, int dbl_halo,
    int flat_h, int flat_w,             // flat mode: input fragments of flat_h x flat_w (0: spatial tiles)
    int dil_h, int dil_w,               // dilated mode (> 1): taps dil apart on one signal, tiled by phase
    int pad_h, int pad_w,               // spatial tiles: a zero border of pad samples around every fragment
    const float* __restrict__ w2,       // kEpiProj: 1x1 projection weights [Cout_pad][4] (binary32, zero padded)
    float* __restrict__ part,           // kEpiProj: partial projections [nbs * WGN][F * Hout * Wout][4]
    int64_t part_stride,                // kEpiProj: floats per channel group of part
    int tile_step_w,                    // columns between neighbouring tiles (TW, or TW - k + 1 with kEpiPool)
    int pool_k, int pool_U) {           // kEpiPool: pool size along the row, pooled samples per fragment
    using Cfg = MfmaCfg<BF16, WGM, WGN, MT, NT>;
    constexpr int THREADS = Cfg::THREADS;
    extern __shared__ __attribute__((aligned(16))) char lds[];
    // The bfloat16 kernel with 128x64 wave tiles keeps its accumulators in the
    // accumulation registers (AGPRs): an AGPR use the compiler cannot rule out
    // (this empty clobber) makes it pick that form of the MFMA instructions.
    // 1 % faster on its longest layers; the narrower bfloat16 tiles and binary32
    // measured slower that way and keep their accumulators in VGPRs.
    if constexpr (BF16 && MT == 4 && NT == 2) asm volatile("" ::: "a0");

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    // The wave index is uniform; held as a scalar it frees the vector registers
    // that its derived values would keep through the K loop (bfloat16 layers
    // 1-4 % faster, binary32 ones 0.4-0.7 %), except in the binary32 kernel
    // with the folded projection, which measured 0.3 % slower that way.
    const int wave = (BF16 || EPI != kEpiProj) ? __builtin_amdgcn_readfirstlane(tid >> 6) : tid >> 6;
    const int wm = wave % WGM;           // wave position along M
    const int wn = wave / WGM;           // wave position along N
    const int half = lane >> 5;          // lane half: K slot of the MFMA operands
    const int l32 = lane & 31;

    // workgroup -> (fragment, tile row, tile column, N block).  Workgroups are
    // handed to the 8 XCDs round-robin by id; the remap gives every XCD one
    // contiguous range of work items.  Items are ordered in groups of kGroup
    // neighbouring tiles (which share halo samples); inside a group the N block
    // is the outer index, so the workgroups that run together on an XCD read the
    // same weight slices and the same input tiles from its L2.
    const int total = gridDim.x;
    const int xcd = blockIdx.x % kXcds, slot = blockIdx.x / kXcds;
    const int q8 = total / kXcds, r8 = total % kXcds;
    const int item = xcd < r8 ? xcd * (q8 + 1) + slot : r8 * (q8 + 1) + (xcd - r8) * q8 + slot;
    const int ntiles = total / nbs;
    const int g = item / (kGroup * nbs);
    const int gsize = min(kGroup, ntiles - g * kGroup);
    const int grem = item - g * kGroup * nbs;
    const int nb = grem / gsize;
    const int tile = g * kGroup + grem % gsize;
    const int tiles = tilesY * tilesX;
    const int f = tile / tiles;
    const int trem = tile % tiles;
    const int ty0 = (trem / tilesX) * TH;
    const int tx0 = (trem % tilesX) * tile_step_w;

    // Spatial tiles: a TH x TW block of one fragment, halo (TH + fh - 1) x (TW + fw - 1).
    // Flat mode (small fragments): the fragment batch is read as one sequence of
    // samples, a tile is TW consecutive positions of it (TH = 1), tap (th, tw)
    // sits th * flat_w + tw samples further on, and only positions that are valid
    // outputs of their own fragment are stored.
    const int HW = flat_w ? TW + (fh - 1) * flat_w + fw - 1 : TW + fw - 1;   // halo row width
    const int tap_row = flat_w ? flat_w : HW;
    const int halo_px = (flat_w ? TH : TH + fh - 1) * HW;
    const int halo_slots = halo_px * kSlotsPerRow;
    const int halo_bytes = ((halo_px * kPitchBytes + 127) / 128) * 128;
    char* halo0 = lds;
    char* halo1 = dbl_halo ? lds + halo_bytes : lds;

    // Tile sample m -> tile row.  An A read (ds_read_b128) is served in four
    // passes of 16 lanes, and on gfx950 the two passes of lanes 0..31 are not
    // lanes 0..15 and 16..31: lane l shares its pass with the lanes whose bits
    // 2, 3 and 4 have the same parity as its own ({0-3, 12-15, 20-27} and the
    // rest; lanes 32..63 alike), which a microbenchmark of two active lanes at
    // conflicting addresses shows.  With the 80-byte sample pitch, halo sample p
    // starts in 16-byte bank group 5p mod 16, and a pass is free of bank
    // conflicts when its 16 samples fall in 16 different groups.  Row-major
    // order achieves that for tiles 32 or more samples wide.  An 8-wide tile
    // puts the 32 samples of an MFMA block on 4 rows, a 16-wide tile on 2; these
    // rows are conflict-free when they are d apart with HW * d = 8 (mod 16) for
    // 8-wide tiles and HW * d = 0 (mod 16) for 16-wide ones.  So such tiles take
    // the groups of TW samples of each block from rows d = 2^row_lg apart,
    // d = 8 >> (trailing zero bits of HW) (8-wide) or 16 >> (trailing zero bits
    // of HW) (16-wide, HW even; an odd HW has no such d and keeps row-major
    // order, as does d = 1), and the epilogue maps m back the same way.  The
    // 8 blocks of a 256-sample tile form groups of d blocks.
    // bfloat16 kernels use one branch-free form of both orders, row =
    // ((m >> sa) << sb) + ((m >> 5) & mb) + (((m >> log2 TW) & mk) << row_lg)
    // (row-major: sa = log2 TW, sb = mb = mk = 0; rows d apart: sa = 5 + row_lg,
    // sb = grp_lg + row_lg, mb = d - 1, mk = 2^grp_lg - 1, where 2^grp_lg = 32 / TW
    // rows hold a block); binary32 kernels a branch on the (uniform) order, which
    // measured faster there (HD 6x6 layer 0.8 % against 0.3 % faster than
    // row-major), while the branch-free form slowed the small bfloat16 layers
    // less (1 % against 2-3 %).
    static_assert(Cfg::BM == 256, "the row order assumes 8 MFMA blocks of 32 samples per tile");
    const int tw_log2 = __builtin_ctz(TW);   // spatial and dilated tiles are 2^k samples wide
    const int hw_tz = __builtin_ctz(HW);
    const int row_lg = TW == 8 ? 3 - min(3, hw_tz) : TW == 16 && hw_tz >= 1 && hw_tz <= 3 ? 4 - hw_tz : 0;
    const int grp_lg = 5 - tw_log2;          // used only with TW = 8 or 16
    const bool rows_apart = row_lg > 0;
    const int sa = rows_apart ? 5 + row_lg : tw_log2, sb = rows_apart ? grp_lg + row_lg : 0;
    const int mb = rows_apart ? (1 << row_lg) - 1 : 0, mk = rows_apart ? (1 << grp_lg) - 1 : 0;
    const int row_lg_b = rows_apart ? row_lg : -1;   // binary32: -1 selects row-major
    auto tile_dy = [&](int m) -> int {
        if constexpr (BF16) {
            return ((m >> sa) << sb) + ((m >> 5) & mb) + (((m >> tw_log2) & mk) << row_lg);
        } else {
            if (row_lg_b < 0) return m >> tw_log2;
            const int blk = m >> 5;
            return (((blk >> row_lg_b) << grp_lg) << row_lg_b) + (blk & ((1 << row_lg_b) - 1)) +
                   (((m & 31) >> tw_log2) << row_lg_b);
        }
    };
    // per-lane operand offsets (bytes) inside the halo / weight slice
    int a_off[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
        const int m = wm * 32 * MT + mt * 32 + l32;
        a_off[mt] = (tile_dy(m) * HW + (m & (TW - 1))) * kPitchBytes + half * 32;
    }

    floatx16 acc[MT][NT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[mt][nt][v] = 0.f;

    const size_t row_bytes = (size_t)Cin * Cfg::ES;
    // Where the tile's halo lives.  Spatial tiles: fragment f, rows and columns
    // adjacent.  Dilated mode: the "fragments" are the dil_h x dil_w phases of one
    // signal; phase (py, px) holds samples (py + dil_h a, px + dil_w b), so a tap
    // step is dil samples and every tile reads and writes one phase only.
    const bool dilated = dil_h * dil_w > 1;
    const int py = dilated ? f / dil_w : 0, px = dilated ? f - py * dil_w : 0;
    const size_t row_step = (size_t)(dilated ? dil_h : 1) * Win * row_bytes;
    const size_t col_step = (size_t)(dilated ? dil_w : 1) * row_bytes;
    const size_t f_base = dilated ? ((size_t)py * Win + px) * row_bytes : (size_t)f * Hin * Win * row_bytes;
    const int lim_h = dilated ? (Hin - py + dil_h - 1) / dil_h : Hin;   // samples of this phase / fragment
    const int lim_w = dilated ? (Win - px + dil_w - 1) / dil_w : Win;
    // top-left input sample of the tile's halo (negative inside the zero border)
    const int hy0 = ty0 - pad_h, hx0 = tx0 - pad_w;
    const char* in_f = in + f_base;
    const int taps = fh * fw;
    const int steps = nchunks * taps;
    const char* w_nb = wp + (size_t)nb * steps * (Cfg::BN * kChunkBytes);
    const char* zero = reinterpret_cast<const char*>(g_zero16);

    // Staging: LDS slot S (16 bytes) of the halo holds quad S % 5 of halo sample
    // S / 5 (slot 4 of every sample is padding and is never written); lane l of
    // wave w stages slot r * THREADS + w * 64 + l in round r.  A round moves S on
    // by THREADS = 51 * 5 + 1 slots, i.e. 51 samples and one quad, so the sample's
    // halo row and column are divided out once and then advanced by additions.
    static_assert(THREADS % kSlotsPerRow == 1, "the slot walk assumes THREADS = 1 mod 5");
    constexpr int kPxStep = THREADS / kSlotsPerRow;
    const int px_first = tid / kSlotsPerRow, q_first = tid - px_first * kSlotsPerRow;
    const int dy_first = px_first / HW, dx_first = px_first - dy_first * HW;
    const int dy_step = kPxStep / HW, dx_step = kPxStep - dy_step * HW;
    // fn(r0, q, yy, xx) for every staged slot of this thread: round base r0, quad
    // q, input sample (yy, xx) of the fragment / phase (negative in the border)
    auto for_each_slot = [&](auto&& fn) {
        int q = q_first, dy = dy_first, dx = dx_first;
        for (int r0 = 0; r0 < halo_slots; r0 += THREADS) {
            if (r0 + tid < halo_slots && q < 4) fn(r0, q, hy0 + dy, hx0 + dx);
            dy += dy_step;
            dx += dx_step;
            if (++q == kSlotsPerRow) {
                q = 0;
                ++dx;
            }
            if (dx >= HW) {
                dx -= HW;
                ++dy;
            }
        }
    };
    auto stage_halo = [&](int cc, char* dst) {
        const char* src_c = in_f + (size_t)cc * kChunkBytes;
        const int c_base = cc * Cfg::CC;
        for_each_slot([&](int r0, int q, int yy, int xx) {
            const bool ok = (unsigned)yy < (unsigned)lim_h && (unsigned)xx < (unsigned)lim_w &&
                            c_base + q * (16 / Cfg::ES) < Cin;
            dma16(ok ? src_c + (size_t)yy * row_step + (size_t)xx * col_step + q * 16 : zero,
                  dst + (r0 + wave * 64) * 16);
        });
    };
    auto wait_staged = [] {
        __builtin_amdgcn_s_waitcnt(0);   // this wave's copies have landed in LDS
        __syncthreads();                 // ... and every other wave's
    };

    // Operand B comes straight from the packed weights in global memory
    // (every workgroup of the N block reads the same slices, which stay in
    // L2) into registers, two steps ahead: no LDS slice and no barrier per
    // step, only one per chunk for the halo.  Lane (n, half) holds bytes
    // 32 half .. 32 half + 31 of row n of a slice (two 16-byte loads), as its
    // halo reads of A do; the slices are packed in lane order (see
    // pack_lane_order), so each load instruction reads one contiguous kilobyte.
    const char* w_lane = w_nb + (size_t)(wn * NT) * kSliceBlock + lane * 16;
    auto load_b = [&](int st, u32x4 (&bb)[NT][2]) {
        const char* src = w_lane + (size_t)st * (Cfg::BN * kChunkBytes);
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int s = 0; s < 2; ++s)
                bb[nt][s] = *reinterpret_cast<const u32x4*>(src + nt * kSliceBlock + s * (kSliceBlock / 2));
    };
    // One step: this tap's A operands from the halo, then the step's MFMAs with
    // the B operands bb (per wave 16 bfloat16 or 64 binary32 issues).  The
    // compiler interleaves the reads with the MFMAs; issuing all eight reads
    // ahead of the first MFMA measured 5 % slower (bfloat16).
    auto mma_step = [&](const char* halo, int tap_off, const u32x4 (&bb)[NT][2]) {
        u32x4 a[2][MT];
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
                a[s][mt] = *reinterpret_cast<const u32x4*>(halo + a_off[mt] + tap_off + 16 * s);
        // bfloat16 kEpiProj computes the transposed block (weights first)
        constexpr bool TR = EPI == kEpiProj && BF16;
        if constexpr (BF16) {
#pragma unroll
            for (int s = 0; s < 2; ++s)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int nt = 0; nt < NT; ++nt)
                        acc[mt][nt] = TR ? __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                                               as_bf16x8(bb[nt][s]), as_bf16x8(a[s][mt]), acc[mt][nt], 0, 0, 0)
                                         : __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                                               as_bf16x8(a[s][mt]), as_bf16x8(bb[nt][s]), acc[mt][nt], 0, 0, 0);
        } else {
#pragma unroll
            for (int s = 0; s < 8; ++s)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int nt = 0; nt < NT; ++nt) {
                        const float av = __uint_as_float(a[s >> 2][mt][s & 3]);
                        const float bv = __uint_as_float(bb[nt][s >> 2][s & 3]);
                        acc[mt][nt] = TR ? __builtin_amdgcn_mfma_f32_32x32x2f32(bv, av, acc[mt][nt], 0, 0, 0)
                                         : __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, acc[mt][nt], 0, 0, 0);
                    }
        }
    };
    // The next chunk's halo is staged by the same copies as stage_halo, but
    // issued as inline assembly.  To the compiler, LDS-DMA completes out of
    // order with ordinary loads, so with one in flight that it knows of,
    // every wait for a B operand would become a wait for all loads; unseen,
    // they leave those waits partial.  The hardware counts them in issue order
    // with the B loads (a partial wait that the compiler computes without
    // them still covers its own loads), and the full wait before the chunk's
    // closing barrier drains them.  M0 (the LDS destination) is saved and
    // restored around each copy.
    const uint32_t lds_base = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;
    auto stage_halo_unseen = [&](int cn, char* dst) {
        const char* src_c = in_f + (size_t)cn * kChunkBytes;
        const int c_base = cn * Cfg::CC;
        const uint32_t dst_lds = lds_base + (uint32_t)(dst - lds);
        for_each_slot([&](int r0, int q, int yy, int xx) {
            const bool ok = (unsigned)yy < (unsigned)lim_h && (unsigned)xx < (unsigned)lim_w &&
                            c_base + q * (16 / Cfg::ES) < Cin;
            const char* src = ok ? src_c + (size_t)yy * row_step + (size_t)xx * col_step + q * 16 : zero;
            const uint32_t m0v = __builtin_amdgcn_readfirstlane(dst_lds + (uint32_t)(r0 + wave * 64) * 16);
            uint32_t saved;
            asm volatile(
                "s_mov_b32 %0, m0\n\t"
                "s_mov_b32 m0, %2\n\t"
                "s_nop 0\n\t"
                "global_load_lds_dwordx4 %1, off\n\t"
                "s_mov_b32 m0, %0"
                : "=&s"(saved)
                : "v"(src), "s"(m0v)
                : "memory");
        });
    };
    // B operands two steps ahead in three register sets whose roles rotate
    // with the step, over all steps of all chunks in threes, so no register
    // copy waits for a load (the loads past the last step repeat the last
    // slice).  A chunk ends inside the rotation: its closing drain and barrier
    // leave the next chunk's halo in place, and the copies of the one after
    // it go out.
    u32x4 bA[NT][2], bB[NT][2], bC[NT][2];
    load_b(0, bA);
    load_b(min(1, steps - 1), bB);
    stage_halo(0, halo0);
    wait_staged();
    if (dbl_halo && nchunks > 1) stage_halo_unseen(1, halo1);
    int step = 0, cc = 0, th = 0, tw = 0;   // step, chunk and tap of the next step
    const char* halo = halo0;
    auto next_chunk = [&]() {
        if (++cc >= nchunks) return;
        if (!dbl_halo) {
            __syncthreads();               // every wave is done with the previous chunk's halo
            stage_halo(cc, halo0);
        }
        wait_staged();                     // chunk cc's halo has landed, for every wave
        halo = (cc & 1) ? halo1 : halo0;
        // chunk cc + 1 goes to the buffer of chunk cc - 1, which every wave is done with
        if (dbl_halo && cc + 1 < nchunks) stage_halo_unseen(cc + 1, (cc & 1) ? halo0 : halo1);
    };
    auto sub_step = [&](const u32x4 (&bb)[NT][2], u32x4 (&bl)[NT][2]) {
        load_b(min(step + 2, steps - 1), bl);
        mma_step(halo, (th * tap_row + tw) * kPitchBytes, bb);
        ++step;
        if (++tw == fw) {
            tw = 0;
            if (++th == fh) {
                th = 0;
                next_chunk();
            }
        }
    };
    while (step + 2 < steps) {
        sub_step(bA, bC);
        sub_step(bB, bA);
        sub_step(bC, bB);
    }
    if (step < steps) sub_step(bA, bC);
    if (step < steps) sub_step(bB, bA);

    // -- epilogue: D[i][j] of a 32x32 tile sits in lane j + 32*((i/4)%2), register (i/8)*4 + i%4
    const int n_base = nb * Cfg::BN + wn * 32 * NT;
    const size_t f_off = (size_t)f * Hout * Wout;
    const int frag_px = flat_h * flat_w;
    // output sample of tile position m: whether it exists, and its index
    auto out_pos = [&](int m, size_t& o) -> bool {
        if (flat_w) {
            const int p = tx0 + m;                 // TH = 1: position in the flat sequence (Win long)
            const int fr = p / frag_px, r = p - fr * frag_px;
            const int y = r / flat_w, x = r - y * flat_w;
            o = ((size_t)fr * Hout + y) * Wout + x;
            return p < Win && y < Hout && x < Wout;
        }
        if (dilated) {
            const int y = py + dil_h * (ty0 + tile_dy(m)), x = px + dil_w * (tx0 + (m & (TW - 1)));
            o = (size_t)y * Wout + x;
            return y < Hout && x < Wout;
        }
        const int y = ty0 + tile_dy(m), x = tx0 + (m & (TW - 1));
        o = f_off + (size_t)y * Wout + x;
        return y < Hout && x < Wout;
    };
    int ncol[NT];
    float bn[NT];
#pragma unroll
    for (int nt = 0; nt < NT; ++nt) {
        ncol[nt] = n_base + nt * 32 + l32;
        bn[nt] = ncol[nt] < Cout ? bias[ncol[nt]] : 0.f;
    }
    // The stores of one activation (a compile-time constant, so the per-value
    // code has no branch on it).
    auto store_tile = [&](auto act_c) {
        constexpr int ACT = decltype(act_c)::value;
        if constexpr (sizeof(Tout) == 2) {
            // bfloat16 output: each lane holds one channel of 16 positions, so direct
            // stores would be 2-byte stores, one instruction per value.  Transpose
            // through LDS (the halo buffers are free now) into 16-byte units of 8
            // channels of one position: 8x fewer store instructions.
            if (Cout % 8 == 0 && ((uintptr_t)out & 15) == 0) {
                constexpr int WCOLS = 32 * NT;                          // channels of a wave's block
                uint16_t* st = reinterpret_cast<uint16_t*>(lds) + wave * (32 * WCOLS);
                __syncthreads();                                        // every wave is done with the halo
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
                    for (int nt = 0; nt < NT; ++nt)
#pragma unroll
                        for (int v = 0; v < 16; ++v) {
                            const int i = (v >> 2) * 8 + half * 4 + (v & 3);
                            st[i * WCOLS + nt * 32 + l32] = f32_to_bf16(activate(ACT, acc[mt][nt][v] + bn[nt]));
                        }
                    // st is this wave's own region and LDS executes a wave's operations
                    // in order: no workgroup barrier between the stores and the loads
                    __builtin_amdgcn_wave_barrier();
#pragma unroll
                    for (int r = 0; r < WCOLS / 16; ++r) {               // 32 rows x WCOLS / 8 units, 64 per round
                        const int u = r * 64 + lane;
                        const int row = u / (WCOLS / 8), c8 = (u % (WCOLS / 8)) * 8;
                        size_t o;
                        if (out_pos(wm * 32 * MT + mt * 32 + row, o) && n_base + c8 < Cout)
                            *reinterpret_cast<u32x4*>(out + o * Cout + n_base + c8) =
                                *reinterpret_cast<const u32x4*>(st + row * WCOLS + c8);
                    }
                    __builtin_amdgcn_wave_barrier();
                }
                return;
            }
        } else {
            // binary32 output: the same transposition, per 32 x 32 block (4.5 KB per
            // wave, within any halo buffer; a 36-float pitch puts the two lane
            // halves' rows in different banks), into 16-byte units of 4 channels:
            // 4x fewer store instructions, each lane-group writing 128 contiguous
            // bytes of one position
            if (Cout % 4 == 0 && ((uintptr_t)out & 15) == 0) {
                constexpr int PITCH = 36;
                float* st = reinterpret_cast<float*>(lds) + wave * (32 * PITCH);
                __syncthreads();                                        // every wave is done with the halo
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
                    for (int nt = 0; nt < NT; ++nt) {
#pragma unroll
                        for (int v = 0; v < 16; ++v) {
                            const int i = (v >> 2) * 8 + half * 4 + (v & 3);
                            st[i * PITCH + l32] = activate(ACT, acc[mt][nt][v] + bn[nt]);
                        }
                        // this wave's own region, LDS operations in order: no workgroup barrier
                        __builtin_amdgcn_wave_barrier();
#pragma unroll
                        for (int r = 0; r < 4; ++r) {                   // 32 rows x 8 units, 64 per round
                            const int u = r * 64 + lane;
                            const int row = u >> 3, c4 = (u & 7) * 4;
                            const int c = n_base + nt * 32 + c4;
                            size_t o;
                            if (out_pos(wm * 32 * MT + mt * 32 + row, o) && c < Cout)
                                *reinterpret_cast<float4*>(out + o * Cout + c) =
                                    *reinterpret_cast<const float4*>(st + row * PITCH + c4);
                        }
                        __builtin_amdgcn_wave_barrier();
                    }
                }
                return;
            }
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
            for (int v = 0; v < 16; ++v) {
                const int i = (v >> 2) * 8 + half * 4 + (v & 3);
                const int m = wm * 32 * MT + mt * 32 + i;
                size_t o;
                bool ok;
                if (flat_w) {
                    const int p = tx0 + m;
                    const int fr = p / frag_px, r = p - fr * frag_px;
                    const int y = r / flat_w, x = r - y * flat_w;
                    ok = p < Win && y < Hout && x < Wout;
                    o = ((size_t)fr * Hout + y) * Wout + x;
                } else if (dilated) {
                    const int y = py + dil_h * (ty0 + tile_dy(m)), x = px + dil_w * (tx0 + (m & (TW - 1)));
                    ok = y < Hout && x < Wout;
                    o = (size_t)y * Wout + x;
                } else {
                    const int y = ty0 + tile_dy(m), x = tx0 + (m & (TW - 1));
                    ok = y < Hout && x < Wout;
                    o = f_off + (size_t)y * Wout + x;
                }
                if (!ok) continue;
#pragma unroll
                for (int nt = 0; nt < NT; ++nt)
                    if (ncol[nt] < Cout)
                        store_elem(out + o * Cout + ncol[nt], activate(ACT, acc[mt][nt][v] + bn[nt]));
            }
        }
    };
    // The following 1x1 convolution folded into this epilogue (kEpiProj): per output
    // sample and projection channel o (four, zero padded), the partial dot
    // product over each wave's group of 32 NT channels (64 with the 64- and
    // 128-channel N tiles, 32 with the 32-channel one),
    //   part[group][sample][o] = sum_{n in group} w2[n][o] * act(acc[sample][n] + bias[n]),
    // summed over the groups in order, with the projection's bias and activation,
    // by the step that reads it.  The groups do not depend on the N tile of the
    // launch, so every evaluation fashion sums in the same order.
    //
    // binary32 (store_proj_lanes): a lane holds one channel of 16 samples per
    // 32x32 tile; per sample it first adds its NT channels' products, then the
    // lanes of a half are reduced in two passes of 8 samples x 4 outputs by five
    // butterfly exchanges that halve the values a lane keeps (32 -> 1), so in
    // pass p lane l32 ends with output o = l32 mod 4 of sample slot v = 8 p + l32 / 4.
    auto store_proj_lanes = [&](auto act_c) {
        constexpr int ACT = decltype(act_c)::value;
        // keeps the projection weights' loads here: hoisted above the K loop they
        // would hold registers through it
        asm volatile("" ::: "memory");
        float4 wv[NT];
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
            wv[nt] = ncol[nt] < Cout ? *reinterpret_cast<const float4*>(w2 + 4 * (size_t)ncol[nt])
                                     : make_float4(0.f, 0.f, 0.f, 0.f);
        // the wave's position as scalars: when the vector wm / wn feed the K
        // loop's addresses, sharing them would keep those values live through it
        const int wm_s = __builtin_amdgcn_readfirstlane(wm), wn_s = __builtin_amdgcn_readfirstlane(wn);
        float* part_g = part + (size_t)(nb * WGN + wn_s) * part_stride;
        const int oc = l32 & 3;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
            for (int pass = 0; pass < 2; ++pass) {
                float v32[32];
#pragma unroll
                for (int v = 0; v < 8; ++v) {
                    float p0 = 0.f, p1 = 0.f, p2 = 0.f, p3 = 0.f;
#pragma unroll
                    for (int nt = 0; nt < NT; ++nt) {
                        const float a = activate(ACT, acc[mt][nt][8 * pass + v] + bn[nt]);
                        p0 += a * wv[nt].x;
                        p1 += a * wv[nt].y;
                        p2 += a * wv[nt].z;
                        p3 += a * wv[nt].w;
                    }
                    v32[4 * v] = p0;
                    v32[4 * v + 1] = p1;
                    v32[4 * v + 2] = p2;
                    v32[4 * v + 3] = p3;
                }
#pragma unroll
                for (int lvl = 0; lvl < 5; ++lvl) {
                    const int sh = 16 >> lvl, n = 16 >> lvl;   // partner lane ^ sh; keep n of 2n values
                    const bool upper = (l32 & sh) != 0;
#pragma unroll
                    for (int t = 0; t < n; ++t) {
                        const float give = upper ? v32[t] : v32[t + n];
                        const float keep = upper ? v32[t + n] : v32[t];
                        v32[t] = keep + __shfl_xor(give, sh, 64);
                    }
                }
                const int vv = 8 * pass + (l32 >> 2);
                const int m = wm_s * 32 * MT + mt * 32 + (vv >> 2) * 8 + half * 4 + (vv & 3);
                size_t o;
                if (out_pos(m, o)) part_g[o * 4 + oc] = v32[0];
            }
        }
    };
    // bfloat16 (store_proj): the kernel computes the transposed 32x32 blocks
    // (the MFMAs take the weights as their first operand), so D[i][j], i a
    // channel and j a sample, sits in lane j + 32*((i/4)%2), register
    // (i/8)*4 + i%4: a lane holds one sample and, in its register group
    // g = v/4, the four consecutive channels 8g + 4*half .. +3.  A lane adds the
    // products of its 16 NT channels of its sample (columns nt, then register
    // groups, then the group's channels, in order), and one exchange between
    // the lane halves (v_permlane32_swap) adds the other 16 NT: the lower half's
    // sum first, outputs 0 and 1 in the lower lane and 2 and 3 in the upper one.
    // On the 4K frame's 6x6 layer that ran 4.7-5.9 % faster than the butterfly
    // form; the binary32 HD frame's 6x6 layer ran 0.3 % slower with it.
    auto store_proj = [&](auto act_c) {
        constexpr int ACT = decltype(act_c)::value;
        // The lane's position again, from the lane-id instructions: the values
        // computed at entry feed the K loop, and sharing them would keep them
        // live through it.
        const int lane_e = __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u));
        const int ll = lane_e & 31, lh = lane_e >> 5;
        const int p_base = nb * Cfg::BN + wn * 32 * NT;
        // Loads from the read-only kernel arguments are invariant to the
        // compiler, which may move them anywhere, up to before the K loop, where
        // their registers would stay live through it: an opaque zero added to
        // the pointer per use keeps each load in its place.
        auto pinned = [](const float* q) {
            int zero = 0;
            asm volatile("" : "+s"(zero));
            return q + zero;
        };
        // first channel of register group g of accumulator column nt (a multiple
        // of 4; bias and w2 hold at least p_base + 32 NT rows)
        auto group_chan = [&](int nt, int g) { return p_base + nt * 32 + g * 8 + lh * 4; };
        auto bias4 = [&](int nt, int g) {
            return *reinterpret_cast<const float4*>(pinned(bias) + group_chan(nt, g));
        };
        float ps[MT][4];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
            for (int o = 0; o < 4; ++o) ps[mt][o] = 0.f;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                // One register group at a time: its weights, then its values.
                // Each value passes through an (empty) ordered asm statement, so
                // the activations cannot all be computed up front, where their
                // results would not fit beside the accumulators.
                const int c = group_chan(nt, g);
                const float4 b = bias4(nt, g);
                const float bv[4] = {b.x, b.y, b.z, b.w};
                const float* w2g = pinned(w2);
                float4 wq[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) wq[u] = *reinterpret_cast<const float4*>(w2g + 4 * (size_t)(c + u));
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int u = 0; u < 4; ++u) {
                        float x = acc[mt][nt][4 * g + u];
                        asm volatile("" : "+v"(x));
                        const float a = activate(ACT, x + bv[u]);
                        ps[mt][0] += a * wq[u].x;
                        ps[mt][1] += a * wq[u].y;
                        ps[mt][2] += a * wq[u].z;
                        ps[mt][3] += a * wq[u].w;
                    }
                // ... and the group's sums are complete before the next group's values
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                    for (int o = 0; o < 4; ++o) asm volatile("" : "+v"(ps[mt][o]));
            }
        float* part_g = part + (size_t)(nb * WGN + wn) * part_stride;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            size_t o;
            const bool ok = out_pos(wm * 32 * MT + mt * 32 + ll, o);
            const auto r0 = __builtin_amdgcn_permlane32_swap(__float_as_uint(ps[mt][0]), __float_as_uint(ps[mt][2]),
                                                             false, false);
            const auto r1 = __builtin_amdgcn_permlane32_swap(__float_as_uint(ps[mt][1]), __float_as_uint(ps[mt][3]),
                                                             false, false);
            // lower lanes hold (own, partner's) sums of outputs 0 and 1, upper
            // lanes (partner's, own) of outputs 2 and 3: the lower half first
            const float2 val = make_float2(__uint_as_float(r0[0]) + __uint_as_float(r0[1]),
                                           __uint_as_float(r1[0]) + __uint_as_float(r1[1]));
            if (ok) *reinterpret_cast<float2*>(part_g + o * 4 + 2 * lh) = val;
        }
    };
    // kEpiPool (fragments of one row, binary32, one wave column): per group of
    // 32 channels (one accumulator column of every wave) the tile's activations
    // go to LDS as [BM][32 + 4] floats (37 KB: with the halo buffers, three
    // workgroups still fit a CU); each thread then forms the maxima of k
    // consecutive samples for the tile's first TW - k + 1 positions
    // (neighbouring tiles overlap by k - 1 samples, so every window lies inside
    // one tile) and writes each maximum straight to its fragment: sample x of
    // input fragment f goes to sample x div k of fragment (x mod k) F + f, F the
    // launch's fragment count (Lemma "frag-ops" along the row).
    auto store_pool = [&](auto act_c) {
        constexpr int ACT = decltype(act_c)::value;
        constexpr int PITCH = 32 + 4;
        constexpr int CQ = 32 / 4;
        float* tl = reinterpret_cast<float*>(lds);
        const int nfrag = ntiles / tilesX;                       // fragments of the launch (tilesY = 1)
        const int npos = TW - pool_k + 1;
#pragma unroll
        for (int nt = 0; nt < NT; ++nt) {
            __syncthreads();                                     // the halo / the previous group is done with
#pragma unroll
            for (int mt = 0; mt < MT; ++mt)
#pragma unroll
                for (int v = 0; v < 16; ++v) {
                    const int m = wm * 32 * MT + mt * 32 + (v >> 2) * 8 + half * 4 + (v & 3);
                    tl[m * PITCH + l32] = activate(ACT, acc[mt][nt][v] + bn[nt]);
                }
            __syncthreads();
            for (int idx = tid; idx < npos * CQ; idx += THREADS) {
                const int pp = idx / CQ, cq = idx - pp * CQ;
                const int x = tx0 + pp;                          // first sample of the window
                const int c0 = n_base + nt * 32 + cq * 4;
                if (x >= pool_k * pool_U || c0 >= Cout) continue;
                float4 mx = *reinterpret_cast<const float4*>(tl + pp * PITCH + cq * 4);
                for (int t = 1; t < pool_k; ++t) {
                    const float4 q = *reinterpret_cast<const float4*>(tl + (pp + t) * PITCH + cq * 4);
                    mx.x = fmaxf(mx.x, q.x);
                    mx.y = fmaxf(mx.y, q.y);
                    mx.z = fmaxf(mx.z, q.z);
                    mx.w = fmaxf(mx.w, q.w);
                }
                const size_t fo = (size_t)(x % pool_k) * nfrag + f;
                *reinterpret_cast<float4*>(reinterpret_cast<float*>(out) + (fo * pool_U + x / pool_k) * Cout + c0) =
                    mx;
            }
        }
    };
    if constexpr (EPI == kEpiPool) {
        if (act == 1)
            store_pool(std::integral_constant<int, 1>{});
        else if (act == 2)
            store_pool(std::integral_constant<int, 2>{});
        else
            store_pool(std::integral_constant<int, 0>{});
        return;
    }
    if constexpr (EPI == kEpiProj) {
        auto proj = [&](auto act_c) {
            if constexpr (BF16) store_proj(act_c);
            else store_proj_lanes(act_c);
        };
        if (act == 1)
            proj(std::integral_constant<int, 1>{});
        else if (act == 2)
            proj(std::integral_constant<int, 2>{});
        else
            proj(std::integral_constant<int, 0>{});
        return;
    }
    if (act == 1)
        store_tile(std::integral_constant<int, 1>{});
    else if (act == 2)
        store_tile(std::integral_constant<int, 2>{});
    else
        store_tile(std::integral_constant<int, 0>{});
}

// ------------------------------------------------------------------ host side

int mfma_f32_pick_bn(int cout) { return cout >= 128 ? 128 : cout >= 64 ? 64 : 32; }
int mfma_bf16_pick_bn(int cout) { return cout >= 128 ? 128 : cout >= 64 ? 64 : 32; }

static size_t packed_elems(const PlanConv& pc, int cc) {
    return (size_t)(pc.cout_pad / pc.bn) * (pc.cin_pad / cc) * pc.fh * pc.fw * pc.bn * cc;
}
size_t mfma_f32_packed_floats(const PlanConv& pc) { return packed_elems(pc, 16); }
size_t mfma_bf16_packed_elems(const PlanConv& pc) { return packed_elems(pc, 32); }

// Each slice in the order the kernel's lanes load it: row n = 32 g + r and the
// channel at byte offset cb = 32 half + 16 s + b of the row's 64-byte chunk go to
// byte ((2 g + s) * 64 + 32 half + r) * 16 + b, the 16-byte operand of lane
// 32 half + r for load s of 32-row block g, so the 64 lanes of one load read
// 1 KB of consecutive bytes.
template <typename E, typename Conv>
static void pack_lane_order(const PlanConv& pc, const float* w, E* dst, Conv conv) {
    constexpr int cc = kChunkBytes / (int)sizeof(E);
    static_assert(32 * kChunkBytes == kSliceBlock, "slice layout");
    const int nbs = pc.cout_pad / pc.bn, nch = pc.cin_pad / cc;
    const size_t slice = (size_t)pc.bn * cc;
    size_t base = 0;
    for (int nb = 0; nb < nbs; ++nb)
        for (int ch = 0; ch < nch; ++ch)
            for (int th = 0; th < pc.fh; ++th)
                for (int tw = 0; tw < pc.fw; ++tw, base += slice)
                    for (int nl = 0; nl < pc.bn; ++nl)
                        for (int cl = 0; cl < cc; ++cl) {
                            const int o = nb * pc.bn + nl, i = ch * cc + cl;
                            float v = 0.f;
                            if (o < pc.cout && i < pc.cin) v = w[(((size_t)o * pc.cin + i) * pc.fh + th) * pc.fw + tw];
                            const int g = nl / 32, r = nl % 32, cb = cl * (int)sizeof(E);
                            const int hf = cb / 32, s = (cb / 16) % 2, b = cb % 16;
                            dst[base + (((size_t)(2 * g + s) * 64 + 32 * hf + r) * 16 + b) / sizeof(E)] = conv(v);
                        }
}

void mfma_f32_pack(const PlanConv& pc, const float* w, float* dst) {
    pack_lane_order(pc, w, dst, [](float v) { return v; });
}
void mfma_bf16_pack(const PlanConv& pc, const float* w, uint16_t* dst) {
    pack_lane_order(pc, w, dst, [](float v) { return host_f32_to_bf16(v); });
}

struct Tile {
    int TH, TW;
    size_t lds;
    int dbl;    // halo double-buffered
};

// Spatial tile TH x TW = BM output samples: the shape that wastes the fewest
// masked samples on this layer's fragment extent; among those, one whose halo can
// be double-buffered within the LDS budget of two workgroups per CU, then the
// smallest halo.  The bfloat16 kernel counts the work of an 8-wide tile whose
// halo row is not 8 mod 16 samples long 3 % higher: such tiles once took LDS
// bank conflicts on their A reads (8 x 32 -> 16 x 16 tiles made the 3x3 layers
// of the 4K frame 18 % faster, while 16 x 16 tiles with 3.4 % more masked work
// made its 6x6 layer 4.7 % slower).  The kernel now reads 8- and 16-wide tiles
// with their rows interleaved (tile_dy); the weight stays: the layers where it
// decides have under 0.3 % of masked work between the two shapes, and 16 x 16
// stages a smaller halo.
static Tile pick_tile(int BM, int Hout, int Wout, int fh, int fw, size_t lds_max, bool bf16) {
    Tile best{0, 0, 0, 0};
    int64_t best_work = -1, best_halo = -1;
    for (int TW = 8; TW <= BM; TW *= 2) {
        const int TH = BM / TW;
        const int64_t halo_px = (int64_t)(TH + fh - 1) * (TW + fw - 1);
        const size_t halo_b = (size_t)((halo_px * kPitchBytes + 127) / 128) * 128;
        const size_t cap = std::min(lds_max, (size_t)kMaxLds);
        int dbl;
        size_t lds;
        if (2 * halo_b <= cap) { dbl = 1; lds = 2 * halo_b; }
        else if (halo_b <= cap) { dbl = 0; lds = halo_b; }
        else continue;
        int64_t work = ceil_div64(Hout, TH) * TH * ceil_div64(Wout, TW) * TW;
        if (bf16 && TW < 16 && (TW + fw - 1) % 16 != 8) work += work / 32;
        const bool better = best_work < 0 || work < best_work ||
                            (work == best_work && (dbl > best.dbl || (dbl == best.dbl && halo_px < best_halo)));
        if (better) {
            best = Tile{TH, TW, lds, dbl};
            best_work = work;
            best_halo = halo_px;
        }
    }
    return best;
}

// Whether some spatial tile fits an fh x fw filter's halo into LDS (checked
// against the 64 KB every device offers).
bool mfma_supports(bool bf16, int fh, int fw) {
    return pick_tile(256, 1, 1, fh, fw, 64 * 1024, bf16).TH > 0 && pick_tile(256, 64, 64, fh, fw, 64 * 1024, bf16).TH > 0;
}

// Flat-mode tile (TH = 1, TW = BM consecutive positions of the flattened
// fragment batch) for fragments of Hin x Win input samples, or TH = 0 if its
// single-row halo does not fit.
static Tile flat_tile(int BM, int Win, int fh, int fw, size_t lds_max) {
    const int64_t halo_px = BM + (int64_t)(fh - 1) * Win + fw - 1;
    const size_t halo_b = (size_t)((halo_px * kPitchBytes + 127) / 128) * 128;
    const size_t cap = std::min(lds_max, (size_t)kMaxLds);
    if (2 * halo_b <= cap) return Tile{1, BM, 2 * halo_b, 1};
    if (halo_b <= cap) return Tile{1, BM, halo_b, 0};
    return Tile{0, 0, 0, 0};
}

// The grid of one launch: a spatial tile per fragment (per phase when dilated),
// or the flat reading of the whole fragment batch when that computes at least
// 10 % fewer positions (small fragments waste most of a spatial tile; the flat
// sequence computes Hin*Win positions per fragment, of which only the last
// fh-1 rows and fw-1 columns are discarded).
struct LaunchShape {
    Tile t;
    int flat;
    int tilesY, tilesX;
    int64_t nblocks;    // 0 if no tile fits
};

// Hin x Win: the fragment extent including any zero border (which rules out the
// flat reading, allow_flat = false).
static LaunchShape launch_shape(int BM, bool bf16, int F, int Hin, int Win, int dil_h, int dil_w, int fh, int fw,
                                int nbs, bool allow_flat = true) {
    LaunchShape L{Tile{0, 0, 0, 0}, 0, 0, 0, 0};
    const size_t lds = device_lds_limit();
    if (dil_h * dil_w > 1) {
        const int Hout = Hin - dil_h * (fh - 1), Wout = Win - dil_w * (fw - 1);
        const int Hp = (int)ceil_div64(Hout, dil_h), Wp = (int)ceil_div64(Wout, dil_w);
        L.t = pick_tile(BM, Hp, Wp, fh, fw, lds, bf16);
        if (L.t.TH == 0) return L;
        L.tilesY = (int)ceil_div64(Hp, L.t.TH);
        L.tilesX = (int)ceil_div64(Wp, L.t.TW);
        L.nblocks = (int64_t)dil_h * dil_w * L.tilesY * L.tilesX * nbs;
        return L;
    }
    const int Hout = Hin - fh + 1, Wout = Win - fw + 1;
    L.t = pick_tile(BM, Hout, Wout, fh, fw, lds, bf16);
    const int64_t flat_len = (int64_t)F * Hin * Win;
    if (allow_flat && flat_len < (1ll << 30)) {
        const Tile ft = flat_tile(BM, Win, fh, fw, lds);
        const int64_t work_tiles =
            L.t.TH ? (int64_t)F * ceil_div64(Hout, L.t.TH) * L.t.TH * ceil_div64(Wout, L.t.TW) * L.t.TW : -1;
        const int64_t work_flat = ceil_div64(flat_len, BM) * BM;
        if (ft.TH && (work_tiles < 0 || 10 * work_flat < 9 * work_tiles)) {
            L.t = ft;
            L.flat = 1;
            L.tilesY = 1;
            L.tilesX = (int)ceil_div64(flat_len, ft.TW);
            L.nblocks = (int64_t)L.tilesX * nbs;
            return L;
        }
    }
    if (L.t.TH == 0) return L;
    L.tilesY = (int)ceil_div64(Hout, L.t.TH);
    L.tilesX = (int)ceil_div64(Wout, L.t.TW);
    L.nblocks = (int64_t)F * L.tilesY * L.tilesX * nbs;
    return L;
}

// The 128-channel N tile or the 64-channel one for a launch.  A launch of fewer
// workgroups than the 512 that the GPU holds at once (two per CU) leaves CUs
// idle or half-loaded; the 64-channel tile doubles the workgroup count at a
// cost of about 10 % per MFMA in operand traffic (measured on the conv6x6
// 256->512 layer of a 135 x 240 fragment).  With every workgroup resident, the
// busiest CU sets the time: ceil(blocks / 256) workgroups of the 128-channel
// tile against ceil(blocks64 / 256) of half the work each.  A lone workgroup
// per CU (one wave per SIMD) hides no MFMA latency, so up to 256 workgroups
// the 64-channel tile is taken.
PlanConv mfma_launch_variant(const PlanConv& pc, int F, int Hin, int Win, int dil_h, int dil_w, int pad_h,
                             int pad_w) {
    if (!pc.w_alt || pc.impl == CONV_DIRECT) return pc;
    const bool bf16 = pc.impl == CONV_MFMA_BF16;
    const bool flat = pad_h == 0 && pad_w == 0;
    Hin += 2 * pad_h;
    Win += 2 * pad_w;
    const LaunchShape a = launch_shape(256, bf16, F, Hin, Win, dil_h, dil_w, pc.fh, pc.fw,
                                       pc.cout_pad / pc.bn, flat);
    if (a.nblocks == 0 || a.nblocks >= 512) return pc;
    const LaunchShape b =
        launch_shape(256, bf16, F, Hin, Win, dil_h, dil_w, pc.fh, pc.fw,
                     pc.cout_pad_alt / pc.bn_alt, flat);
    if (b.nblocks == 0) return pc;
    if (a.nblocks > 256 && 11 * ceil_div64(b.nblocks, 256) >= 20 * ceil_div64(a.nblocks, 256)) return pc;
    PlanConv alt = pc;
    alt.w = pc.w_alt;
    alt.bn = pc.bn_alt;
    alt.cout_pad = pc.cout_pad_alt;
    return alt;
}

int mfma_tile_mode(const PlanConv& pc, int F, int Hin, int Win, int dil_h, int dil_w, int pad_h, int pad_w) {
    if (pc.impl == CONV_DIRECT) return -1;
    if (dil_h * dil_w > 1) return 2;
    const bool padded = pad_h > 0 || pad_w > 0;
    const LaunchShape L = launch_shape(256, pc.impl == CONV_MFMA_BF16, F, Hin + 2 * pad_h, Win + 2 * pad_w, dil_h,
                                       dil_w, pc.fh, pc.fw, pc.cout_pad / pc.bn, !padded);
    return L.flat ? 1 : 0;
}

template <bool BF16, typename Tout, int WGM, int WGN, int MT, int NT, int EPI>
static hipError_t run_mfma(const void* in, int F, int Hin, int Win, int dil_h, int dil_w, int pad_h, int pad_w,
                           const PlanConv& pc, void* out, float* part, int pool_k, hipStream_t s) {
    using Cfg = MfmaCfg<BF16, WGM, WGN, MT, NT>;
    const bool dilated = dil_h * dil_w > 1;
    const bool padded = pad_h > 0 || pad_w > 0;
    if (dilated && F != 1) return hipErrorInvalidValue;   // dilated: one signal, tiled per phase
    if (padded && (dilated || pad_h < 0 || pad_w < 0)) return hipErrorInvalidValue;
    const int nbs = pc.cout_pad / Cfg::BN;
    LaunchShape L = launch_shape(Cfg::BM, BF16, F, Hin + 2 * pad_h, Win + 2 * pad_w, dil_h, dil_w, pc.fh, pc.fw, nbs,
                                 !padded);
    if (L.nblocks == 0) return hipErrorInvalidConfiguration;
    // A single channel chunk reads one halo: the second buffer would only halve
    // the workgroups that fit a CU.
    if (pc.cin_pad == Cfg::CC && L.t.dbl) {
        L.t.dbl = 0;
        L.t.lds /= 2;
    }
    // kEpiPool: spatial tiles of one row of BM samples, stepped by BM - k + 1
    // columns, and LDS for the tile's activations
    int tile_step_w = L.t.TW, pool_U = 0;
    if constexpr (EPI == kEpiPool) {
        const int Wout = Win - pc.fw + 1;
        if (BF16 || WGN != 1 || dil_h * dil_w > 1 || pad_h || pad_w || Hin != pc.fh || pool_k < 2 ||
            pool_k >= Cfg::BM || (Wout - pool_k + 1) % pool_k != 0 || pc.cout % 4 != 0)
            return hipErrorInvalidValue;
        pool_U = (Wout - pool_k + 1) / pool_k;
        tile_step_w = Cfg::BM - pool_k + 1;
        const int64_t halo_b = ((int64_t)pc.fh * (Cfg::BM + pc.fw - 1) * kPitchBytes + 127) / 128 * 128;
        if (halo_b > kMaxLds) return hipErrorInvalidValue;
        L.t = Tile{1, Cfg::BM, (size_t)halo_b, 0};
        if (pc.cin_pad > Cfg::CC && 2 * halo_b <= kMaxLds) {
            L.t.dbl = 1;
            L.t.lds = 2 * halo_b;
        }
        L.t.lds = std::max(L.t.lds, (size_t)Cfg::BM * (32 + 4) * sizeof(float));
        L.flat = 0;
        L.tilesY = 1;
        L.tilesX = (int)ceil_div64((int64_t)pool_k * pool_U, tile_step_w);
        L.nblocks = (int64_t)F * L.tilesX * nbs;
    }
    if (L.nblocks >= (1ll << 31)) return hipErrorInvalidConfiguration;
    auto kern = conv_mfma_kernel<BF16, Tout, WGM, WGN, MT, NT, EPI>;
    hipError_t e = allow_dynamic_lds((const void*)kern, L.t.lds);
    if (e != hipSuccess) return e;
    const int nchunks = pc.cin_pad / Cfg::CC;
    const int Hout = Hin + 2 * pad_h - dil_h * (pc.fh - 1), Wout = Win + 2 * pad_w - dil_w * (pc.fw - 1);
    if (EPI == kEpiProj && (padded || !pc.w2)) return hipErrorInvalidValue;
    const int64_t part_stride = EPI == kEpiProj ? (int64_t)F * Hout * Wout * 4 : 0;
    if (L.flat) {
        // one "fragment" of 1 x (F * Hin * Win) samples for the staging and the tile grid
        const int flat_len = (int)((int64_t)F * Hin * Win);   // below 2^30 in flat mode
        kern<<<dim3((unsigned)L.nblocks), Cfg::THREADS, L.t.lds, s>>>(
            (const char*)in, 1, flat_len, pc.cin, (const char*)pc.w, pc.b, pc.fh, pc.fw, pc.cout, pc.act, nchunks,
            (Tout*)out, Hout, Wout, 1, L.t.TW, 1, L.tilesX, nbs, L.t.dbl, Hin, Win, 1, 1, 0, 0, pc.w2, part,
            part_stride, L.t.TW, 0, 0);
        return hipGetLastError();
    }
    kern<<<dim3((unsigned)L.nblocks), Cfg::THREADS, L.t.lds, s>>>(
        (const char*)in, Hin, Win, pc.cin, (const char*)pc.w, pc.b, pc.fh, pc.fw, pc.cout, pc.act, nchunks,
        (Tout*)out, Hout, Wout, L.t.TH, L.t.TW, L.tilesY, L.tilesX, nbs, L.t.dbl, 0, 0, dil_h, dil_w, pad_h, pad_w,
        pc.w2, part, part_stride, tile_step_w, pool_k, pool_U);
    return hipGetLastError();
}

template <bool BF16, typename Tout, int EPI = kEpiStore>
static hipError_t dispatch_bn(const void* in, int F, int Hin, int Win, int dh, int dw, int ph, int pw,
                              const PlanConv& pc, void* out, hipStream_t s, float* part = nullptr, int pool_k = 0) {
    switch (pc.bn) {
        case 128:
            if constexpr (EPI == kEpiPool) return hipErrorInvalidValue;   // one wave column only
            else return run_mfma<BF16, Tout, 2, 2, 4, 2, EPI>(in, F, Hin, Win, dh, dw, ph, pw, pc, out, part, 0, s);
        case 64: return run_mfma<BF16, Tout, 4, 1, 2, 2, EPI>(in, F, Hin, Win, dh, dw, ph, pw, pc, out, part, pool_k, s);
        case 32: return run_mfma<BF16, Tout, 4, 1, 2, 1, EPI>(in, F, Hin, Win, dh, dw, ph, pw, pc, out, part, pool_k, s);
    }
    return hipErrorInvalidValue;
}

hipError_t launch_conv_mfma_f32(const float* in, int F, int Hin, int Win, int dil_h, int dil_w, const PlanConv& pc,
                                float* out, hipStream_t s) {
    return dispatch_bn<false, float>(in, F, Hin, Win, dil_h, dil_w, 0, 0, pc, out, s);
}

hipError_t launch_conv_mfma_f32_padded(const float* in, int F, int Hin, int Win, int pad_h, int pad_w,
                                       const PlanConv& pc, float* out, hipStream_t s) {
    return dispatch_bn<false, float>(in, F, Hin, Win, 1, 1, pad_h, pad_w, pc, out, s);
}

hipError_t launch_conv_mfma_bf16(dss_dtype tout, const uint16_t* in, int F, int Hin, int Win, int dil_h, int dil_w,
                                 const PlanConv& pc, void* out, hipStream_t s) {
    if (tout == DSS_F32) return dispatch_bn<true, float>(in, F, Hin, Win, dil_h, dil_w, 0, 0, pc, out, s);
    return dispatch_bn<true, uint16_t>(in, F, Hin, Win, dil_h, dil_w, 0, 0, pc, out, s);
}

hipError_t launch_conv_mfma_proj(const void* in, int F, int Hin, int Win, int dil_h, int dil_w, const PlanConv& pc,
                                 float* part, hipStream_t s) {
    if (pc.impl == CONV_MFMA_BF16)
        return dispatch_bn<true, float, kEpiProj>(in, F, Hin, Win, dil_h, dil_w, 0, 0, pc, nullptr, s, part);
    if (pc.impl == CONV_MFMA_F32)
        return dispatch_bn<false, float, kEpiProj>(in, F, Hin, Win, dil_h, dil_w, 0, 0, pc, nullptr, s, part);
    return hipErrorInvalidValue;
}

hipError_t launch_conv_mfma_pool(const float* in, int F, int Hin, int Win, const PlanConv& pc, int pool_k, float* out,
                                 hipStream_t s) {
    if (pc.impl != CONV_MFMA_F32) return hipErrorInvalidValue;
    return dispatch_bn<false, float, kEpiPool>(in, F, Hin, Win, 1, 1, 0, 0, pc, out, s, nullptr, pool_k);
}

}  // namespace dss
