// Implicit-GEMM convolution on the fp32 matrix cores (v_mfma_f32_16x16x4_f32).
//
// The convolution is the product D = A * B with
//   A [C_out x C_in*K*K]  = the weights (OIHW as they are, or prepacked),
//   B [C_in*K*K x pixels] = input patches, never materialised: every B element
//                           is read from a zero-padded input halo tile in LDS,
//   D [C_out x pixels]    = the NCHW output.
//
// How the ILP-M ideas (Section 4, Algorithm 2) land on CDNA4:
//  * Lanes own output channels for the weight operand.  In a 16x16x4 MFMA the
//    lane (g, l) supplies A[l][g], i.e. the weight of output channel l for
//    channel g of the step -- so each lane loads the filter values of "its"
//    output channel straight from global memory into registers, the paper's
//    filter_reg, with no shared-memory copy of the weights.  In OIHW the K*K
//    taps of one (output, input) channel pair are contiguous, so a lane
//    fetches them with 16-byte loads; the prepacked layout makes every such
//    load instruction of a wave one contiguous kilobyte.  They are loaded one
//    stage ahead, a few instructions per step of the current stage.
//  * The input tile is staged once in LDS for the whole workgroup, by DMA
//    (buffer loads that write LDS directly), and read by every wavefront:
//    lanes own output pixels for the B operand.
//  * Between two barriers a wavefront runs a long barrier-free stream of
//    independent matrix instructions (1024 multiply-adds each), every operand
//    reused by a row or a column of accumulator blocks.
//
// Contraction order.  Within a stage of CC input channels the contraction
// index runs tap-major, channel-minor: MFMA step (t, c4) covers tap t and the
// channel group c4 (4 channels, one per 16-lane group).  Any order of the
// sum is the same convolution; this one makes every LDS address a per-lane
// base plus a compile-time offset.
//
// Work split inside a workgroup: NWC x NWP x NWK wavefronts.  Wave (wc, wp, wk)
// owns 16*MA output channels (slab wc), NB blocks of 16 pixels (group wp) and
// the channel groups wk, wk + NWK, ... of every stage; the NWK partial
// accumulators of a tile are summed through LDS at the end.
//
// Work split across workgroups: output tiles (TH x TW pixels x COT channels)
// and, optionally, `splits` contiguous ranges of input-channel stages.  With
// splits > 1 (or a pooled epilogue) each workgroup writes its partial output,
// in the output's own layout, to slice `split` of the workspace.  The slices
// are summed in split order, so the result does not depend on the order in
// which workgroups run: by the last of a tile's workgroups to finish (fused
// finish: a per-tile arrival count, no second launch), or by a second kernel
// (the pooled epilogue, and on request).
//
// LDS: two stage buffers of the halo [CC][HR][HCP] -- (TH-1)*S+K rows of
// (TW-1)*S+K pixels -- laid out so that the four channel groups of a step
// read different banks (see Cfg).//
// This header holds the kernel templates and what the host side needs of
// them; the compiled variants are instantiated in conv_igemm_v*.hip (several
// files, so that they compile in parallel) and the host side -- plans,
// launches, the split-sum and packing kernels -- is conv_igemm.hip.
#pragma once

#include <cmath>
#include <cstdint>
#include <type_traits>
#include <utility>

#include "internal.h"

namespace ilpm {
namespace ig {

// Unsigned division by a divisor d >= 1 fixed at launch, for dividends below
// 2^31: q = (mulhi(n, m) + n) >> l with l = ceil(log2 d) and
// m = floor(2^32 (2^l - d) / d) + 1 (Granlund and Montgomery, "Division by
// invariant integers using multiplication", 1994, Section 4).  The sum stays
// below 2^32 because mulhi(n, m) < n.  Three scalar instructions instead of
// the ~30 of a general division, which matter in a set-up issued by one wave
// per SIMD.
struct FastDiv {
    unsigned d, m, l;
};

inline FastDiv make_fastdiv(unsigned d)
{
    unsigned l = 0;
    while ((1ull << l) < d) ++l;
    const uint64_t m = (((1ull << l) - d) << 32) / d + 1;
    return FastDiv{d, (unsigned)m, l};
}

__device__ __forceinline__ unsigned fast_div(unsigned n, const FastDiv &f) { return (__umulhi(n, f.m) + n) >> f.l; }

struct IgArgs {
    int c_in, h, w, c_out, pad, h_out, w_out;
    int nchunks, chunks_per_split;
    FastDiv ntiles, co_tiles, tiles_w;  // workgroup -> (split, output-channel tile, spatial tile)
    FastDiv sp_tiles;                    // spatial tiles (tiles_h * tiles_w)
    int sp_fast;  // consecutive workgroups take consecutive spatial tiles (else output-channel tiles)
    int to_part;  // write raw partial sums to slice `split` of the workspace
    int relu;     // otherwise: store max(conv + bias, 0)
    int splits;   // input-channel splits (workgroups per output tile)
    int fuse;     // to_part: the tile's last workgroup sums the slices into out (with ReLU)
    int pool_tile;  // out is the 2x2 max-pooled output, pooled in the workgroup (PoolTile)
};

// One compiled kernel variant: its configuration and a launcher.
struct Variant {
    const char *name;
    int ks, s, th, tw, nwc, nwp, nwk, ma, cc;
    int nt, cot, lds;
    int stages;  // 0: any number of stages per workgroup; else exactly this many
    bool wl;     // weights through LDS: reads OIHW, and its prepacked weights are an OIHW copy
    int nbuf;    // stage buffers
    bool pf;     // progressive first stage: needs at least two stages per workgroup
    bool poolable;  // has a PoolTile instantiation (2x2 max-pool in the workgroup)
    bool c1;        // consecutive channels per lane (Cfg::C1): plans need C_in a multiple of 4
    void (*launch)(dim3 grid, hipStream_t st, const float *, const float *, const float *, float *, float *,
                   const IgArgs &, bool packed);
};

// The variant table, in parts (conv_igemm_v*.hip): each sets *table and
// returns its length.
int variants_part0(const Variant **table);
int variants_part1(const Variant **table);
int variants_part2(const Variant **table);
int variants_part3(const Variant **table);
int variants_part4(const Variant **table);
int variants_part5(const Variant **table);
int variants_part6(const Variant **table);
int variants_part7(const Variant **table);
int variants_part8(const Variant **table);
int variants_part9(const Variant **table);
int variants_part10(const Variant **table);

}  // namespace ig

namespace {

using ig::fast_div;
using ig::FastDiv;
using ig::IgArgs;
using ig::make_fastdiv;
using ig::Variant;


typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void *lds_ptr_t;

constexpr int round64(int n) { return (n + 63) / 64 * 64; }
constexpr int cmax(int a, int b) { return a > b ? a : b; }

template <int KS_, int S_, int TH_, int TW_, int NWC_, int NWP_, int NWK_, int MA_, int CC_, int NBUF_ = 2, int NS_ = 0,
          bool WL_ = false, bool PF_ = false>
struct Cfg {
    static constexpr int KS = KS_, S = S_, TH = TH_, TW = TW_;
    static constexpr int NWC = NWC_, NWP = NWP_, NWK = NWK_, MA = MA_, CC = CC_;
    // Stage buffers: 2 = the next stage's loads fly during this stage; 3 =
    // the loads of the stage after next, for stages shorter than a memory
    // round trip (small tiles).
    static constexpr int NBUF = NBUF_;
    static_assert(NBUF >= 2 && NBUF <= 6, "two to six stage buffers");
    // More than two buffers: the kernel is built for exactly NS stages per
    // workgroup, so its stage sequence is straight-line code with no exits
    // (which keeps the compiler's own tracking of the loads in flight exact:
    // a loop or an early exit merges its state and it then waits on loads
    // the stage does not need).
    static constexpr int NS = NS_;
    static_assert(NBUF == 2 ? NS == 0 : NS >= 1, "a deeper pipeline needs a fixed stage count");
    static constexpr int NW = NWC * NWP * NWK;  // wavefronts per workgroup
    static constexpr int NT = 64 * NW;
    static constexpr int NPIX = TH * TW;
    static constexpr int NB = (NPIX + 16 * NWP - 1) / (16 * NWP);
    static constexpr int KK = KS * KS;
    static constexpr int HR = (TH - 1) * S + KS;
    static constexpr int HC = (TW - 1) * S + KS;
    // A 16 x 16 halo (14 x 14 tiles, 3x3, stride 1) is stored with unpadded
    // 16-word rows, so one DMA instruction fills four whole rows of one
    // channel and a wave always fills the same four rows (QUAD): its lanes'
    // offsets are computed once and stepped by a channel plane.  Each plane
    // is then padded by 16 words, which puts the four channel groups of an
    // MFMA step on different LDS banks (with 256-word planes they share
    // banks, and the stages run ~25% slower).  Other halos pad the rows.
    static constexpr bool QUAD = S == 1 && HC == 16 && HR == 16 && NW % 4 == 0;
    // Other halos are stored unpadded (HCP = HC, PL = HR*HC).  Against a bank
    // model of gfx950's LDS fitted to hardware counters (32 banks of 4 bytes,
    // a ds_read_b32 served as two half-waves of 32 lanes, one pass per
    // distinct word a bank holds in a half), these tight layouts cost at most
    // two extra passes per B read, and layouts padded to make the reads
    // conflict-free measured slower (ResNet conv4.x 7.25 us padded, 6.75 us
    // tight; the strided layer 5.95 / 5.31; the 5x5 layer 13.08 / 12.57): the
    // padding is halo DMA the small-tile kernels wait on, while a conflict
    // adds a pass to reads issued steps ahead.  The 16x16 halo (14x14 tiles)
    // keeps 16-word rows for its four-rows-per-instruction DMA, and with
    // 14-pixel rows in them every 16-pixel block spans two rows: two of its
    // banks hold a word of each of the half-wave's two channels whatever the
    // plane pitch, one extra pass per half on 12 of the 13 blocks.
    static constexpr int HCP = QUAD ? 16 : HC;
    static constexpr int PL = QUAD ? HR * HCP + 16 : HR * HC;  // channel plane stride
    static constexpr int COT = NWC * 16 * MA;
    // A tile of 16*q + t pixels, t in 1..4, computes its last pixel block with
    // the 4x4x1 matrix instruction (16 blocks of 4 channels x 4 pixels, one k
    // each), a quarter of the 16x16x4 one's cycles: block b = 4*kq + cg of
    // lane l = 16*kq + 4*cg + j takes channels 4*cg..4*cg+3 of the 16, k-slice
    // kq of the step's 4 and pixel j -- the same A register as the 16x16x4
    // layout -- and the four k-slice partials are summed across lane groups
    // at the end.
    static constexpr int TAILP = NPIX % 16;
    static constexpr bool TAIL4 = NWP == 1 && TAILP >= 1 && TAILP <= 4;
    // A 4x4x1 instruction placed between 16x16x4 ones occupies the matrix
    // pipe as long as a 16x16x4; back to back they issue about every 9.5
    // cycles.  So a stage's tail instructions run as one burst after its
    // 16x16x4 work, spread over four accumulators (acc[m][NB-1+j], j < 4,
    // folded into acc[m][NB-1] at the end) to keep them independent.
    static constexpr int NBM = TAIL4 ? NB - 1 : NB;  // 16x16x4 blocks
    static constexpr int NACC = TAIL4 ? NB + 3 : NB;
    static constexpr int G4 = CC / 4 / NWK;  // channel groups per wave per stage
    // Which channel of a stage lane (g, l) of wave wk takes in its channel
    // group c4.  In general 4*wk + g + 4*NWK*c4 (the four lane groups of a
    // step on four neighbouring channel planes).  For 1x1 filters with a
    // multiple of four groups per lane (C1) the lane's channels are
    // consecutive instead, G4*(4*wk + g) + c4, so that four of its OIHW
    // weights are one 16-byte load (with the interleaved order each is a
    // 4-byte load, 16 output-channel rows per instruction; plans of these
    // variants need C_in a multiple of 4, so that no such load crosses the
    // end of the tensor).  The B reads and the prepacked layout follow the
    // same order.
    static constexpr bool C1 = KS == 1 && G4 % 4 == 0 && !WL_ && !PF_;
    static constexpr int LSTEP = C1 ? G4 : 1;       // planes between lanes' channels (ci_lane = 4*wk + g)
    static constexpr int CSTEP = C1 ? 1 : 4 * NWK;  // planes between a lane's channel groups
    // One stage buffer: the halo, a whole number of 64-word rows (one DMA
    // instruction each).
    static constexpr int XSZ = round64(CC * PL);
    // DMA instructions per stage: QUAD, four per channel (rows 4q..4q+3 of
    // channel c to LDS word c*PL + 64q); otherwise one per 64 LDS words.
    static constexpr int NIX = QUAD ? CC * HR / 4 : XSZ / 64;
    static constexpr int XPT = (NIX + NW - 1) / NW;  // DMA instructions per wave
    __device__ static constexpr int dma_dst(int e) { return QUAD ? (e / (HR / 4)) * PL + (e % (HR / 4)) * 64 : e * 64; }
    // Weights through LDS (WL): instead of each lane gathering its own
    // weights from OIHW (16 different rows per load instruction, which with
    // small tiles leaves every stage waiting on the L1), a stage's weight
    // block -- COT output channels x CC input channels x KK taps -- is copied
    // after the halo by 16-byte-per-lane DMA of contiguous OIHW runs: input
    // channel c at plane c*CPL, output channel r at row r*KKP within it, taps
    // padded to KKP = KK rounded up to 4, so a 4-tap piece never mixes
    // channels.  The matrix instructions read their A operands from LDS four
    // taps at a time (ds_read_b128), lane (g, l) at plane g, row l: a KKP-word
    // row pitch and a plane pitch COT*KKP, a multiple of 64 words, measured
    // conflict-free on gfx950 (a 12- or 28-word pitch puts the 16 lanes of a
    // plane on 16 disjoint 4-bank groups); the earlier layout, rows of
    // CC*KKP+4 words with channels 12 words apart, took 4 extra passes per
    // read.  Piece j of a run holds taps 4j..4j+3, except the last
    // one (j = NJ-1), which holds the run's last four taps KK-4..KK-1: every
    // 16-byte load then lies inside its own (output, input) channel pair's
    // run, so no load reaches past the run, let alone past the tensor.
    static constexpr bool WL = WL_;
    static_assert(!WL || KK >= 4, "weights through LDS need runs of at least one whole piece");

    static constexpr int KKP = (KK + 3) / 4 * 4;
    static constexpr int NJ = KKP / 4;  // 4-tap pieces per run
    // First tap of piece j, and where tap t lies within its piece t / 4.
    __host__ __device__ static constexpr int piece_tap0(int j) { return j < NJ - 1 ? 4 * j : KK - 4; }
    __host__ __device__ static constexpr int piece_pos(int t) { return t - piece_tap0(t / 4); }
    static constexpr int CPL = COT * KKP;  // weight plane per input channel: a multiple of 64 words
    static constexpr int NIXW = WL ? (CC * CPL + 255) / 256 : 0;  // weight DMA instructions (64 lanes x 4 words)
    static constexpr int WSZ = WL ? NIXW * 256 : 0;
    static constexpr int SBUF = XSZ + WSZ;  // one stage buffer: halo, then weights
    // LDS for the cross-wave sum of the NWK partial accumulators.
    static constexpr int RED = (NWK - 1) * NWC * NWP * MA * NB * 4 * 64;
    static constexpr int BUF0 = cmax(SBUF, RED);
    // The last stage streamed: computed a group of SGB pixel blocks at a time
    // (see compute_stage_streamed).  With the input channels split over
    // waves (NWK > 1) and more than one group, each group's partials are
    // summed across the waves as soon as the group is done (SSPLIT), through
    // an LDS area of their own (the stage buffer is still being read),
    // double-buffered by group: SSLOTS block slots (the group's blocks and,
    // with group 0, the tail's) per wave and group.  Without that split a
    // group is one block: its stores start after the first block and trail
    // the matrix work by one block (VGG-early 64->64 at 224^2 with device-
    // scope stores: 29.2 us, against 29.9 with groups of three).
    static constexpr int SGB = NWK > 1 ? (NBM >= 9 ? 3 : 4) : 1;
    static constexpr bool SSPLIT = NWK > 1 && NBM > SGB;
    static constexpr int SSLOTS = SGB + (TAIL4 ? 1 : 0);
    static constexpr int PARKS = SSPLIT ? 2 * (NWK - 1) * NWC * NWP * MA * SSLOTS * 4 * 64 : 0;
    // Progressive first stage (PF): the first stage's halo goes to buffers of
    // its own, one per group of four channels (GSZ words each), and its
    // weights to registers group by group, so that its matrix work starts
    // once the first group has landed instead of the whole stage.  Every
    // workgroup issues its first loads at the same moment, so that first
    // stage is bound by the memory system's bandwidth, not its latency.
    static constexpr bool PF = PF_;
    static_assert(!PF || (QUAD && NW == 4 && NWK == 1 && MA == 1 && !WL && NBUF == 2 && G4 >= 2 && G4 <= 4),
                  "progressive first stage: four-row halo DMA, one channel group per wave, two buffers");
    static constexpr int GSZ = 4 * PL;
    static constexpr int LDS_BYTES = (BUF0 + (NBUF - 1) * SBUF + (PF ? G4 * GSZ : 0) + PARKS) * 4;
    static_assert(!SSPLIT || (NBUF == 2 && NWP == 1), "the streamed split last stage follows a two-buffer loop");
    static_assert(CC % (4 * NWK) == 0, "a stage holds whole groups of 4 channels per wave");
    static_assert(LDS_BYTES <= 160 * 1024, "LDS budget of one compute unit");
    static_assert(NT <= 1024, "workgroup size");
    // Cache policy of the kernel's own stores (the output, or the partial
    // sums of a split plan), of the final sums a self-summing split writes
    // (OPOL), and whether the workgroups of a tile finish the split sum
    // themselves (see FusedSplit).
    static constexpr int SPOL = 0;
    static constexpr int OPOL = 0;
    static constexpr bool FUSED = false;
    // A 2x2 max-pool can be applied inside the workgroup (PoolTile) when the
    // tile's windows do not cross tiles (even TH, TW) and the tile's outputs
    // fit in LDS beside the stage buffers.
    static constexpr bool POOL = false;
    static constexpr bool STREAM_POOL = false;
    static constexpr int POOL_FLOATS = COT * NPIX;
    static constexpr bool POOLABLE =
        TH % 2 == 0 && TW % 2 == 0 && LDS_BYTES - 4 * PARKS + 4 * POOL_FLOATS <= 160 * 1024;
};

// The same configuration for split plans whose tiles sum their own partial
// sums (finish_split_tile).  The partial sums are stored at device scope
// (cache policy SC1: written through to where the XCDs' L2 caches are
// coherent) and read back at device scope, so the workgroup that sums a tile
// sees the other XCDs' slices without writing back or invalidating whole L2
// caches.
constexpr int kPolicyDeviceScope = 16;  // SC1 in a buffer instruction's cache-policy operand
template <class C>
struct FusedSplit : C {
    static constexpr int SPOL = kPolicyDeviceScope;
    static constexpr bool FUSED = true;
};

// The same configuration for split plans whose partial sums a second kernel
// adds (sum_splits, sum_splits_pool): the partial sums are stored at device
// scope, written through each XCD's L2 while the kernel runs instead of
// being written back from the L2 caches when it ends (512->512 at 28^2 in
// eight splits: 38.0 -> 33.3 us).
template <class C>
struct SplitPart : C {
    static constexpr int SPOL = kPolicyDeviceScope;
};

// The same configuration with the output stores at device scope (SC1):
// written through each XCD's L2 while the kernel runs rather than written
// back from the L2 caches when it ends, which overlaps moving a large output
// into memory with the matrix work of the last stage.
template <class C>
struct Sc1Out : C {
    static constexpr int SPOL = kPolicyDeviceScope;
    static constexpr int OPOL = kPolicyDeviceScope;
};

// The same configuration with the 2x2 max-pool epilogue done in the
// workgroup: the last stage writes its results (ReLU applied, when asked) to
// an LDS copy of the tile instead of the output, in the same order and with
// the same values, and pool_tile_finish writes the maxima of the tile's 2x2
// windows.  The result is that of conv -> ReLU -> pool, without writing the
// full-size output or launching a second kernel.
template <class C>
struct PoolTile : C {
    static_assert(C::POOLABLE, "pooled tiles need even tile sides and LDS room for the tile");
    static constexpr bool POOL = true;
    // One channel group per wave and every pixel of the tile in each wave:
    // a wave's rows of the LDS tile are its own, so it pools them as they
    // fill, during the streamed last stage (see compute_stage_streamed),
    // with no workgroup barrier.
    static constexpr bool STREAM_POOL = C::NWK == 1 && C::NWP == 1;
};


// Buffer descriptors give branch-free loads: a lane whose element lies in the
// zero padding (or past the tensor) carries an offset beyond the descriptor's
// range and reads 0.  Offsets are bytes and fit in 31 bits (checked when the
// plan is made).
constexpr int kOutOfRange = 0x7fffffff;
constexpr int kBufferWord3 = 0x00020000;  // 32-bit elements, raw (stride 0) buffer

// A descriptor for [base, base + bytes).  Both are wave-uniform; saying so
// explicitly keeps the descriptor in scalar registers (otherwise the compiler
// may build it in vector registers and wrap every load in a loop over the
// distinct values).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const float *base, unsigned bytes)
{
    const uint64_t b = reinterpret_cast<uint64_t>(base);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    float *p = reinterpret_cast<float *>(((uint64_t)hi << 32) | lo);
    return __builtin_amdgcn_make_buffer_rsrc(p, (short)0, (int)__builtin_amdgcn_readfirstlane(bytes), kBufferWord3);
}

// Weight registers of one stage for one lane: [m-block][channel group][tap].
template <class C, bool WL = C::WL>
struct AStage {
    float v[C::MA][C::G4][C::KK];
};

// Weights through LDS: what a lane needs is where its A operands lie, the
// LDS word of (m-block m, channel group 0, tap 0) relative to the stage
// buffer (the same for every stage).
template <class C>
struct AStage<C, true> {
    int base[C::MA];
};

// Where a lane's weights come from.  Every wave holds, per stage, the
// weights of its 16*MA output channels for its channel groups, as
// A.v[m][c4][t] = w[co0 + wc*16*MA + 16*m + l][ci0 + 4*wk + g + 4*NWK*c4][t]
// for lane (g, l) (with Cfg::C1, channel ci0 + G4*(4*wk + g) + c4).  A source issues them as NA single load instructions,
// load(q) being the q-th.
struct WeightCtx {
    __amdgpu_buffer_rsrc_t rw;
    int c_in, nchunks;
    int co_lane0;  // co0 + wc*16*MA + l16 (output channel of m-block 0)
    int ci_lane;   // 4*wk + g
    int block0;    // prepacked layout: (co_t*nchunks)*NWK*NWC + wk*NWC + wc
    int lane;
    int c_out, wave;
    const float *w;     // OIHW weights (weights through LDS)
    const void *wl;     // weights through LDS: this lane's DMA offsets (WlLanes<C>)
};

// OIHW weights: lane (g, l) reads its own contiguous run of KK taps per
// (m, c4), in 16-byte pieces plus 4-byte ones for the tail of the run.
template <class C>
struct OihwWeights {
    static constexpr int kPieces = C::KK / 4 + C::KK % 4;
    // C1: load j*MA + m holds channel groups 4j..4j+3 of m-block m.
    static constexpr int NA = C::C1 ? C::G4 / 4 * C::MA : C::G4 * C::MA * kPieces;
    static constexpr int NA_MIN = NA;  // issued by every wave
    // The last load (in issue order) of channel group c's registers.
    static constexpr int group_last(int c) { return C::C1 ? (c / 4 + 1) * C::MA - 1 : (c + 1) * C::MA * kPieces - 1; }
    __amdgpu_buffer_rsrc_t rw;
    unsigned a_base[C::G4][C::MA];

    __device__ __forceinline__ OihwWeights(const WeightCtx &k, int c_out, int ci0, float *) : rw(k.rw)
    {
        // One row product per m-block, then additions: no branches, and only
        // MA full 32-bit multiplies.
        const unsigned row_b = (unsigned)k.c_in * (C::KK * 4u);
        unsigned row[C::MA];
        bool co_ok[C::MA];
#pragma unroll
        for (int m = 0; m < C::MA; ++m) {
            const int co = k.co_lane0 + 16 * m;
            co_ok[m] = co < c_out;
            row[m] = (unsigned)co * row_b;
        }
#pragma unroll
        for (int c4 = 0; c4 < C::G4; ++c4) {
            // C1: a_base[j][m] (j < G4/4) for groups 4j..4j+3, all four inside
            // the row or all past it (C_in and the first channel multiples of 4).
            const int ci = C::C1 ? ci0 + k.ci_lane * C::G4 + 4 * c4 : ci0 + k.ci_lane + 4 * C::NWK * c4;
#pragma unroll
            for (int m = 0; m < C::MA; ++m)
                a_base[c4][m] =
                    (ci < k.c_in && co_ok[m]) ? row[m] + (unsigned)ci * (C::KK * 4u) : (unsigned)kOutOfRange;
        }
    }

    __device__ __forceinline__ void load(int q, AStage<C> &A) const
    {
        if constexpr (C::C1) {
            const int j = q / C::MA, m = q % C::MA;
            const floatx4 v =
                __builtin_bit_cast(floatx4, __builtin_amdgcn_raw_buffer_load_b128(rw, (int)a_base[j][m], 0, 0));
            A.v[m][4 * j][0] = v[0];
            A.v[m][4 * j + 1][0] = v[1];
            A.v[m][4 * j + 2][0] = v[2];
            A.v[m][4 * j + 3][0] = v[3];
            return;
        }
        const int c4 = q / (C::MA * kPieces), m = (q / kPieces) % C::MA, piece = q % kPieces;
        const unsigned base = a_base[c4][m];
        float *dst = A.v[m][c4];
        if (piece < C::KK / 4) {
            const floatx4 v = __builtin_bit_cast(
                floatx4, __builtin_amdgcn_raw_buffer_load_b128(rw, (int)(base + 16u * piece), 0, 0));
            dst[4 * piece] = v[0];
            dst[4 * piece + 1] = v[1];
            dst[4 * piece + 2] = v[2];
            dst[4 * piece + 3] = v[3];
        } else {
            const int e = C::KK / 4 * 4 + (piece - C::KK / 4);
            dst[e] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rw, (int)(base + 4u * e), 0, 0));
        }
    }
};

// Prepacked weights (ilpm_conv2d_prepack_weights): for each (output-channel
// tile, chunk of CC input channels, wk, wc) one block of 64*EPL floats, EPL =
// MA*G4*KK, holding lane l's A.v in flat order; floats 4i..4i+3 of every lane
// lie together ([i][lane][4]), so load instruction i of a wave reads one
// contiguous kilobyte, and the last EPL mod 4 floats of each lane follow as
// [j][lane] (one 256-byte load each).  Channels past C_out or C_in are
// stored as zeros.
template <class C>
struct PackedWeights {
    static constexpr int EPL = C::MA * C::G4 * C::KK;
    static constexpr int N4 = EPL / 4, REM = EPL % 4;
    static constexpr int NA = N4 + REM;
    static constexpr int NA_MIN = NA;
    // The last load (in issue order) of channel group c's registers (one
    // m-block: group c is elements KK*c .. KK*c + KK - 1).
    static constexpr int group_last(int c)
    {
        const int e = C::KK * (c + 1) - 1;
        return e < 4 * N4 ? e / 4 : N4 + (e - 4 * N4);
    }
    __amdgpu_buffer_rsrc_t rw;
    unsigned base;  // bytes: this wave's block for the stage

    __device__ __forceinline__ PackedWeights(const WeightCtx &k, int, int ci0, float *) : rw(k.rw)
    {
        const int block = k.block0 + (ci0 / C::CC) * C::NWK * C::NWC;
        base = (unsigned)block * (64u * EPL * 4u);
        lane = k.lane;
    }
    int lane;

    // Element e of the lane's flat order is A.v[m][c4][t] with
    // e = (m*G4 + c4)*KK + t.
    __device__ __forceinline__ static void put(AStage<C> &A, int e, float v)
    {
        A.v[e / (C::G4 * C::KK)][(e / C::KK) % C::G4][e % C::KK] = v;
    }

    __device__ __forceinline__ void load(int q, AStage<C> &A) const
    {
        if (q < N4) {
            const floatx4 v = __builtin_bit_cast(
                floatx4, __builtin_amdgcn_raw_buffer_load_b128(rw, (int)(base + 1024u * q + 16u * lane), 0, 0));
#pragma unroll
            for (int j = 0; j < 4; ++j) put(A, 4 * q + j, v[j]);
        } else {
            // Remainder float j = q - N4, one 4-byte load (in this toolchain
            // the 8- and 12-byte buffer-load builtins come out as a single
            // 4-byte load copied into every element, so they are not used).
            const int j = q - N4;
            put(A, 4 * N4 + j,
                __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                              rw, (int)(base + 1024u * N4 + 256u * j + 4u * lane), 0, 0)));
        }
    }
};

// Weights through LDS: per lane and weight DMA instruction j of this wave
// (instruction e = j*NW + wave, 4-word piece 64*e + lane of the weight area),
// the byte offset of its first OIHW element relative to the stage's first
// input channel, or 2^31 for row padding and channels past C_out, and its
// input channel within the stage, which at or past C_in reads nothing.  Each
// piece's 16 bytes lie inside one (output, input) channel pair's KK taps (the
// last piece of a run starts at tap KK-4, see Cfg), so a load is either
// wholly inside the tensor or, at offset 2^31, wholly past the descriptor's
// range, where a buffer load returns zeros.
template <class C>
struct WlLanes {
    static constexpr int XPTW = (C::NIXW + C::NW - 1) / C::NW;
    unsigned off[XPTW];
    int col[XPTW];

    __device__ __forceinline__ void init(int co0, int c_in, int c_out, int wave, int lane)
    {
#pragma unroll
        for (int j = 0; j < XPTW; ++j) {
            const int q = (j * C::NW + wave) * 64 + lane;  // 4-word piece of the weight area
            const int c = q / (C::CPL / 4), rem = q - c * (C::CPL / 4);
            const int r = rem / (C::KKP / 4), piece = rem - r * (C::KKP / 4);
            const int co = co0 + r;
            const bool ok = r < C::COT && c < C::CC && co < c_out;
            off[j] = ok ? (unsigned)(co * c_in * C::KK + c * C::KK + C::piece_tap0(piece)) * 4u : 0x80000000u;
            col[j] = ok ? c : C::CC;  // the piece's input channel within the stage
        }
    }
};

template <class C>
struct LdsWeights {
    static constexpr int XPTW = WlLanes<C>::XPTW;
    static constexpr int kFullW = C::NIXW / C::NW;
    static constexpr int NA = XPTW;
    static constexpr int NA_MIN = kFullW;
    __amdgpu_buffer_rsrc_t rw;
    const WlLanes<C> *lanes;
    float *dst;  // the stage buffer's weight area, after its halo
    int lim;     // C_in - ci0: the stage's input channels that exist
    int wave;

    __device__ __forceinline__ LdsWeights(const WeightCtx &k, int c_out, int ci0, float *buf)
        : lanes(static_cast<const WlLanes<C> *>(k.wl)), dst(buf + C::XSZ), wave(k.wave)
    {
        const int64_t total = (int64_t)c_out * k.c_in * C::KK;
        const int64_t first = (int64_t)ci0 * C::KK;
        rw = make_rsrc(k.w + first, first < total ? (unsigned)(total - first) * 4u : 0u);
        lim = k.c_in - ci0;
    }

    __device__ __forceinline__ void load(int q, AStage<C> &) const
    {
        if (q >= kFullW && q * C::NW + wave >= C::NIXW) return;  // a last, partial round
        const unsigned o = lanes->col[q] < lim ? lanes->off[q] : 0x80000000u;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr_t)(dst + (q * C::NW + wave) * 256), 16, (int)o, 0, 0,
                                                 0);
    }
};

// All of a stage's weights at once (the first stage).
template <class C, class WS>
__device__ __forceinline__ void load_a(AStage<C> &A, const WS &ws)
{
#pragma unroll
    for (int q = 0; q < WS::NA; ++q) ws.load(q, A);
}

// Per-lane offsets of the halo DMA, the same for every stage: DMA instruction
// i of a stage fills LDS words [64*i, 64*i + 64) of the stage buffer, lane l
// word 64*i + l; wave w issues instructions w, w + NW, w + 2*NW, ...
template <class C>
__device__ __forceinline__ void halo_offsets(int (&xo)[C::XPT], const IgArgs &a, int wave, int lane, int ih0,
                                             int iw0)
{
    if constexpr (C::QUAD) {
        // Instruction j of wave w covers channel (j*NW + w)/4, rows 4q..4q+3
        // with q = w % 4: lane l at row 4q + l/16, column l % 16.
        // A lane outside the image starts at 2^31: plus any channel offset
        // (below 2^31) it stays past every descriptor's range.
        const int ih = ih0 + 4 * (wave % 4) + (lane >> 4), iw = iw0 + (lane & 15);
        const bool ok = ih >= 0 && ih < a.h && iw >= 0 && iw < a.w;
        const unsigned base = ok ? (unsigned)(ih * a.w + iw) * 4u : 0x80000000u;
        const unsigned plane = (unsigned)a.h * (unsigned)a.w * 4u;
#pragma unroll
        for (int j = 0; j < C::XPT; ++j) {
            const unsigned c = (unsigned)((j * C::NW + wave) / 4);
            xo[j] = (int)(base + c * plane);
        }
    } else {
#pragma unroll
        for (int j = 0; j < C::XPT; ++j) {
            const int e = (j * C::NW + wave) * 64 + lane;
            const int c = e / C::PL;
            const int rem = e - c * C::PL;
            const int r = rem / C::HCP;
            const int col = rem - r * C::HCP;
            const int ih = ih0 + r, iw = iw0 + col;
            const bool ok = c < C::CC && col < C::HC && ih >= 0 && ih < a.h && iw >= 0 && iw < a.w;
            xo[j] = ok ? ((c * a.h + ih) * a.w + iw) * 4 : kOutOfRange;
        }
    }
}

// The input from channel ci0 on, as a buffer descriptor: channels at or past
// C_in lie past its end and read 0.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t halo_rsrc(const float *__restrict__ x, const IgArgs &a, int ci0)
{
    const unsigned plane = (unsigned)a.h * (unsigned)a.w;
    return make_rsrc(x + (size_t)ci0 * plane, ci0 < a.c_in ? (unsigned)(a.c_in - ci0) * plane * 4u : 0u);
}

// Issue the halo DMA of a stage (descriptor rx from halo_rsrc) into `buf`.
template <class C>
__device__ __forceinline__ void dma_halo(float *buf, const __amdgpu_buffer_rsrc_t &rx, int wave,
                                         const int (&xo)[C::XPT])
{
    constexpr int kFull = C::NIX / C::NW;  // rounds in which every wave issues one
#pragma unroll
    for (int j = 0; j < kFull; ++j)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_ptr_t)(buf + C::dma_dst(j * C::NW + wave)), 4, xo[j], 0, 0,
                                                 0);
    if constexpr (kFull < C::XPT) {
        if (kFull * C::NW + wave < C::NIX)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_ptr_t)(buf + C::dma_dst(kFull * C::NW + wave)), 4,
                                                     xo[kFull], 0, 0, 0);
    }
}

// The loads of the next stage -- its halo DMA and its weight registers --
// as a list of single instructions that compute_stage issues a few at a time
// between its matrix instructions.  Issued in one burst at the start of a
// stage, they fill the memory pipeline's queue and the wave stalls at issue
// with its matrix pipe idle; spread over the stage's steps they drain as
// they go, the last landing while the stage's last steps run.  Item i < ND is
// DMA instruction i of this wave; the rest are the weight loads, one 16-byte
// (or, for the tail of a tap run, 4-byte) piece each.
template <class C, class WS>
struct NextStage {
    static constexpr int kFull = C::NIX / C::NW;
    static constexpr int ND = C::XPT;
    static constexpr int N = ND + WS::NA;

    __amdgpu_buffer_rsrc_t rx;
    float *buf;
    AStage<C> *A;
    const int *xo;
    int wave;
    WS ws;

    __device__ __forceinline__ NextStage(float *buf_, AStage<C> &A_, const float *__restrict__ x, const IgArgs &a,
                                         const WeightCtx &wk, int ci0, int wave_, const int (&xo_)[C::XPT])
        : buf(buf_), A(&A_), xo(xo_), wave(wave_), ws(wk, a.c_out, ci0, buf_)
    {
        const unsigned plane = (unsigned)a.h * (unsigned)a.w;
        // A stage starting at or past C_in gets an empty range: its loads
        // read zeros and touch no memory.
        rx = make_rsrc(x + (size_t)ci0 * plane, ci0 < a.c_in ? (unsigned)(a.c_in - ci0) * plane * 4u : 0u);
    }

    __device__ __forceinline__ void issue(int i)
    {
        if (i < ND) {
            if (i < kFull) {
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_ptr_t)(buf + C::dma_dst(i * C::NW + wave)), 4, xo[i], 0,
                                                         0, 0);
            } else if (kFull * C::NW + wave < C::NIX) {
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_ptr_t)(buf + C::dma_dst(kFull * C::NW + wave)), 4,
                                                         xo[kFull], 0, 0, 0);
            }
            return;
        }
        ws.load(i - ND, *A);
    }
};

// No next stage (the last one).
struct NoNextStage {
    static constexpr int N = 0;
    __device__ __forceinline__ void issue(int) {}
};

// Every load in flight (this wave's DMA and weight registers) has landed, and
// then every wave's.  The wait is the builtin (vmcnt = 0, expcnt and lgkmcnt
// left at their maxima) rather than inline assembly so that the compiler
// knows the loads are complete and adds no waits of its own later.
__device__ __forceinline__ void stage_ready()
{
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();
}

// The same with the K most recent loads of this wave still in flight (the
// stage after next).  Vector-memory loads complete in issue order, so the
// count leaves exactly the older stage's loads landed; K is at most the
// fewest loads any wave issues for a stage.  vmcnt is split over bits 3:0
// and 15:14 of the wait's immediate.
template <int K>
__device__ __forceinline__ void stage_ready_keep()
{
    static_assert(K >= 0 && K < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt(0x0F70 | (K & 15) | ((K >> 4) << 14));
    // A bare barrier: __syncthreads() also orders this wave's pending LDS
    // writes -- the DMA of the stage after next -- before it, which would
    // wait for them.  The data each wave needs next is complete by the count
    // above, and every LDS read of the stage just computed has been consumed
    // by its matrix instructions.  The empty asm statements keep the compiler
    // from moving memory accesses across.
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// The end of a stage of a pipelined plan: its next stage's loads landed,
// with K of the latest still in flight.
template <class C, int K>
__device__ __forceinline__ void stage_wait()
{
    if constexpr (K > 0) {
        stage_ready_keep<K>();
    } else {
        stage_ready();
    }
}

// B fragments (input patches) of step st for one wave.
template <class C>
__device__ __forceinline__ void read_b(const float *xl, const int (&b_base)[C::NB], int st, float (&bv)[C::NB])
{
    const int t = st / C::G4, c4 = st % C::G4;
    const int kh = t / C::KS, kw = t % C::KS;
#pragma unroll
    for (int n = 0; n < C::NB; ++n) bv[n] = xl[b_base[n] + C::CSTEP * c4 * C::PL + kh * C::HCP + kw];
}

// One stage of MFMA work for one wave: every tap, this wave's channel groups,
// all MA x NB accumulator blocks.  The B fragments are software pipelined:
// the LDS reads of step s+D are issued before the matrix instructions of
// step s, and scheduling barriers keep the compiler from sinking them -- a
// wave issues in order, so reads placed behind a run of MFMAs would only
// start once the whole run had issued, leaving the matrix pipe to wait on
// them.  D is one step when a step has three or more matrix instructions
// (their 96+ cycles cover an LDS read); waves with one or two blocks per
// step read two or four steps ahead.
template <class C>
struct BPipe {
    static constexpr int kMf = C::MA * C::NBM;
    static constexpr int kSteps = C::KK * C::G4;
    static constexpr int kWant = kMf >= 3 ? 1 : (kMf == 2 ? 2 : 4);
    static constexpr int D = kWant < kSteps ? kWant : (kSteps > 1 ? kSteps - 1 : 1);
    static constexpr int R = D + 1;  // ring slots
};

template <class C, class P>
__device__ __forceinline__ void compute_stage(const float *xl, const AStage<C> &A, const int (&b_base)[C::NB],
                                              floatx4 (&acc)[C::MA][C::NACC], P &next)
{
    constexpr int kSteps = C::KK * C::G4;
    constexpr int D = BPipe<C>::D, R = BPipe<C>::R;
    // Next-stage loads per step: spread over all of the stage's steps (on
    // the nine-step stages of four-wave channel splits, loads issued within
    // the first half cost ~0.13 us per stage more; within the first quarter
    // or at once, far more: the wave stalls at their issue).
    constexpr int kRate = P::N == 0 ? 1 : (P::N + kSteps - 1) / kSteps;
    float bv[R][C::NB];
    float tb[C::TAIL4 ? kSteps : 1];
    float ta[C::WL && C::TAIL4 ? C::MA : 1][C::WL && C::TAIL4 ? kSteps : 1];  // the tail burst's A (WL)
    // Weights through LDS: the A operands of taps 4j..4j+3 (piece j) for
    // every m-block and channel group, one 16-byte LDS read each, the next
    // piece read while the current one is used.
    constexpr int NJ = C::NJ;
    floatx4 ach[C::WL ? 2 : 1][C::MA][C::WL ? C::G4 : 1];
    auto read_a_piece = [&](int j, int slot) {
        if constexpr (C::WL) {
#pragma unroll
            for (int m = 0; m < C::MA; ++m)
#pragma unroll
                for (int c4 = 0; c4 < C::G4; ++c4)
                    ach[slot][m][c4] =
                        *reinterpret_cast<const floatx4 *>(xl + A.base[m] + c4 * 4 * C::NWK * C::CPL + 4 * j);
        }
    };
    read_a_piece(0, 0);
#pragma unroll
    for (int s = 0; s < D && s < kSteps; ++s) read_b<C>(xl, b_base, s, bv[s]);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
        const int cur = st % R;
        const int t = st / C::G4, c4 = st % C::G4;
        const int j = t / 4;
        const bool piece_read = C::WL && c4 == 0 && t % 4 == 0 && j + 1 < NJ;
#pragma unroll
        for (int r = 0; r < kRate; ++r)
            if (st * kRate + r < P::N) next.issue(st * kRate + r);
        if (piece_read) read_a_piece(j + 1, (j + 1) & 1);
        if (st + D < kSteps) read_b<C>(xl, b_base, st + D, bv[(st + D) % R]);
#pragma unroll
        for (int m = 0; m < C::MA; ++m) {
            float a_op;
            if constexpr (C::WL) a_op = ach[j & 1][m][c4][C::piece_pos(t)];
            else a_op = A.v[m][c4][t];
            if constexpr (C::WL && C::TAIL4) ta[m][st] = a_op;
#pragma unroll
            for (int n = 0; n < C::NBM; ++n)
                acc[m][n] = __builtin_amdgcn_mfma_f32_16x16x4f32(a_op, bv[cur][n], acc[m][n], 0, 0, 0);
        }
        if constexpr (C::TAIL4) tb[st] = bv[cur][C::NB - 1];
        // Within the step: one matrix instruction, then one read of a later
        // step, so the reads issue while the matrix pipe is busy.
        constexpr int kMf = C::MA * C::NBM;
        const int n_ds = (st + D < kSteps ? C::NB : 0) + (piece_read ? C::MA * C::G4 : 0);
#pragma unroll
        for (int i = 0; i < (kMf > C::NB + C::MA * C::G4 ? kMf : C::NB + C::MA * C::G4); ++i) {
            if (i < kMf) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            if (i < n_ds) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (C::TAIL4) {
#pragma unroll
        for (int st = 0; st < kSteps; ++st) {
            const int t = st / C::G4, c4 = st % C::G4;
#pragma unroll
            for (int m = 0; m < C::MA; ++m) {
                float a_op;
                if constexpr (C::WL) a_op = ta[m][st];
                else a_op = A.v[m][c4][t];
                acc[m][C::NB - 1 + st % 4] =
                    __builtin_amdgcn_mfma_f32_4x4x1f32(a_op, tb[st], acc[m][C::NB - 1 + st % 4], 0, 0, 0);
            }
        }
        __builtin_amdgcn_sched_barrier(0);
    }
}

// f(integral_constant<int, I>) for I = 0, 1, ..., in order.
template <class F, int... I>
__device__ __forceinline__ void for_each_index(std::integer_sequence<int, I...>, F &&f)
{
    (f(std::integral_constant<int, I>{}), ...);
}

// Progressive first stage (PF): instruction i < 4 of channel group c's halo
// DMA, channel 4c + i (with four waves, DMA instruction j of a wave is
// channel j), into group c's own buffer.
template <class C>
__device__ __forceinline__ void dma_group(float *gbuf, const __amdgpu_buffer_rsrc_t &rx, int c, int i, int wave,
                                          const int (&xo)[C::XPT])
{
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_ptr_t)(gbuf + i * C::PL + 64 * wave), 4, xo[4 * c + i], 0, 0,
                                             0);
}

// The first stage of a PF plan.  Group 0's loads (halo DMA, then weights)
// were issued before the set-up and have landed; the other groups' loads and
// then the next stage's are issued here, a few per step over the first half
// of the stage.  The steps run group by group (every tap of channel group 0,
// then group 1, ...), and before the first LDS read of group c every wave
// waits for its own loads of that group -- vector-memory loads complete in
// issue order, so the count of loads issued after them, known at compile
// time, is the wait -- and then for the other waves at a barrier.
template <class C, class WS, class P, class GB>
__device__ __forceinline__ void first_stage(const GB &gb, const __amdgpu_buffer_rsrc_t &rx, const WS &ws,
                                            AStage<C> &A, const int (&xo)[C::XPT], int wave,
                                            const int (&b_base)[C::NB], floatx4 (&acc)[C::MA][C::NACC], P &next)
{
    constexpr int kSteps = C::KK * C::G4;
    constexpr int D = BPipe<C>::D, R = BPipe<C>::R;
    static_assert(D < C::KK, "a group's first reads follow its wait");
    static_assert(C::NIX % C::NW == 0 && WS::NA == WS::NA_MIN, "every wave issues every load");
    static_assert(WS::group_last(C::G4 - 1) == WS::NA - 1, "the groups cover the stage's weights");
    // Group c's loads: its 4 DMA instructions, then weight loads
    // group_last(c - 1) + 1 .. group_last(c); done(c) = the loads of groups
    // 0..c (group 0's were issued before the set-up).
    constexpr auto first_w = [](int c) { return c == 0 ? 0 : WS::group_last(c - 1) + 1; };
    constexpr auto done = [](int c) { return 4 * (c + 1) + WS::group_last(c) + 1; };
    constexpr int NG = done(C::G4 - 1) - done(0);
    constexpr int NI = NG + P::N;
    constexpr int kIssueSteps = kSteps / 2;
    constexpr int kRate = (NI + kIssueSteps - 1) / kIssueSteps;
    auto issue = [&](int k) {
        if (k < NG) {
#pragma unroll
            for (int c = 1; c < C::G4; ++c) {
                const int u = k + done(0) - done(c - 1);  // index within group c
                if (u >= 0 && k + done(0) < done(c)) {
                    if (u < 4) dma_group<C>(gb(c), rx, c, u, wave, xo);
                    else ws.load(first_w(c) + (u - 4), A);
                }
            }
        } else if (k < NI) {
            next.issue(k - NG);
        }
    };
    // Loads this wave issued after group c's, at its wait before step
    // c*KK - D: group 0's and those of the steps before.
    auto group_wait = [&](auto cc) {
        constexpr int c = decltype(cc)::value;
        constexpr int w = c * C::KK - D;
        constexpr int issued = done(0) + (w * kRate < NI ? w * kRate : NI);
        static_assert(issued >= done(c), "a group's loads are issued before its wait");
        // At most 63 loads are ever in flight (the counter's width; issue
        // stalls beyond), so with more issued after the group's, waiting for
        // 63 still leaves the group's loads landed.
        stage_ready_keep<(issued - done(c) < 63 ? issued - done(c) : 63)>();
    };
    auto read = [&](int st, float(&bv)[C::NB]) {
        const int c4 = st / C::KK, t = st % C::KK;
        const int kh = t / C::KS, kw = t % C::KS;
        const float *xl = gb(c4);
#pragma unroll
        for (int n = 0; n < C::NB; ++n) bv[n] = xl[b_base[n] + kh * C::HCP + kw];
    };
    float bv[R][C::NB];
    float tb[C::TAIL4 ? kSteps : 1];
#pragma unroll
    for (int st = 0; st < D; ++st) read(st, bv[st]);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int st = 0; st < kSteps; ++st) {
        const int cur = st % R;
        const int c4 = st / C::KK, t = st % C::KK;
        if (st + D < kSteps && (st + D) % C::KK == 0) {
            for_each_index(std::make_integer_sequence<int, 4>{}, [&](auto cc) {
                if constexpr (decltype(cc)::value >= 1 && decltype(cc)::value < C::G4)
                    if ((st + D) / C::KK == decltype(cc)::value) group_wait(cc);
            });
        }
#pragma unroll
        for (int r = 0; r < kRate; ++r) {
            const int k = st * kRate + r;
            issue(k);
            // The waits count loads in issue order: no load of a later group
            // (or of the next stage) may be scheduled before a group's last.
            bool group_end = false;
#pragma unroll
            for (int c = 1; c < C::G4; ++c) group_end |= k + done(0) + 1 == done(c);
            if (group_end) __builtin_amdgcn_sched_barrier(0);
        }
        if (st + D < kSteps) read(st + D, bv[(st + D) % R]);
#pragma unroll
        for (int m = 0; m < C::MA; ++m)
#pragma unroll
            for (int n = 0; n < C::NBM; ++n)
                acc[m][n] = __builtin_amdgcn_mfma_f32_16x16x4f32(A.v[m][c4][t], bv[cur][n], acc[m][n], 0, 0, 0);
        if constexpr (C::TAIL4) tb[st] = bv[cur][C::NB - 1];
        constexpr int kMf = C::MA * C::NBM;
        const int n_ds = st + D < kSteps ? C::NB : 0;
#pragma unroll
        for (int i = 0; i < (kMf > C::NB ? kMf : C::NB); ++i) {
            if (i < kMf) __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            if (i < n_ds) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (C::TAIL4) {
#pragma unroll
        for (int st = 0; st < kSteps; ++st) {
            const int c4 = st / C::KK, t = st % C::KK;
#pragma unroll
            for (int m = 0; m < C::MA; ++m)
                acc[m][C::NB - 1 + st % 4] =
                    __builtin_amdgcn_mfma_f32_4x4x1f32(A.v[m][c4][t], tb[st], acc[m][C::NB - 1 + st % 4], 0, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
    }
}

// Weights through LDS: all of a stage's A operands of this lane, from the
// stage buffer into registers (the last stage of a one-group-per-wave plan
// walks its steps once per pixel group).
template <class C>
__device__ __forceinline__ void load_stage_a(const float *xl, const AStage<C> &A,
                                             float (&av)[C::MA][C::G4][C::KK])
{
#pragma unroll
    for (int m = 0; m < C::MA; ++m)
#pragma unroll
        for (int c4 = 0; c4 < C::G4; ++c4) {
            const float *src = xl + A.base[m] + c4 * 4 * C::NWK * C::CPL;
#pragma unroll
            for (int j = 0; j < C::NJ; ++j) {
                const floatx4 v = *reinterpret_cast<const floatx4 *>(src + 4 * j);
                // The last piece repeats taps the one before holds.
#pragma unroll
                for (int e = 0; e < 4; ++e)
                    if (C::piece_tap0(j) + e >= 4 * j) av[m][c4][C::piece_tap0(j) + e] = v[e];
            }
        }
}

// acc[m][NB-1] = the sum of the four tail accumulators, in a fixed order.
template <class C>
__device__ __forceinline__ void fold_tail(floatx4 (&acc)[C::MA][C::NACC])
{
    if constexpr (C::TAIL4) {
#pragma unroll
        for (int m = 0; m < C::MA; ++m)
            acc[m][C::NB - 1] = (acc[m][C::NB - 1] + acc[m][C::NB]) + (acc[m][C::NB + 1] + acc[m][C::NB + 2]);
    }
}

// Where and how one wave stores its accumulators.
template <class C>
struct Epilogue {
    __amdgpu_buffer_rsrc_t ro;
    unsigned pix_off[C::NB];   // byte offset of each pixel block's lane pixel
    unsigned chan_off[C::MA];  // byte offset of output channel co_lane + 16*m (row 0 of the m-block)
    float b[C::MA][4];
    // The 4x4x1 tail block (TAIL4): after the k-slice sum, lane 4*cg + j of
    // the first 16 stores channels tail_co + 16*m + r, r = 0..3, at pixel j.
    int tail_co, c_out, relu;
    unsigned tail_pix, plane_b;
    // POOL: results go to the LDS tile pl [COT][NPIX] (channel co0 + c at
    // row c); the offsets above then address it in bytes.
    float *pl;
    int pool_co0;
    // STREAM_POOL: the pooled output, its sizes, this tile's first pooled
    // row and column, and this wave's first channel row in the LDS tile.
    __amdgpu_buffer_rsrc_t pro;
    int pool_hp, pool_wpo, pool_pi0, pool_pj0, pool_wc0;

    // RELU: 0 = as the launch says (relu), 1 = no ReLU, 2 = ReLU (the last
    // stage decides once instead of per store).
    template <int RELU = 0>
    __device__ __forceinline__ float fin(float v) const
    {
        const bool on = RELU == 0 ? relu != 0 : RELU == 2;
        return on && v < 0.f ? 0.f : v;
    }

    // Lane channel co_lane + 16*m + r's bias (with partial sums, split 0's
    // carry it and the others none).  A lane's channels past C_out never
    // store, so their bias is read from the last channel instead of being
    // masked.
    __device__ __forceinline__ void load_bias(const IgArgs &a, const float *bias, int co_lane, int split)
    {
#pragma unroll
        for (int m = 0; m < C::MA; ++m)
#pragma unroll
            for (int r = 0; r < 4; ++r) b[m][r] = 0.f;
        if (bias != nullptr && (!a.to_part || split == 0)) {
#pragma unroll
            for (int m = 0; m < C::MA; ++m)
#pragma unroll
                for (int r = 0; r < 4; ++r) b[m][r] = bias[min(co_lane + 16 * m + r, a.c_out - 1)];
        }
    }

    // with_bias = false: load_bias was called already.
    __device__ __forceinline__ void init(const IgArgs &a, float *out, float *part, const float *bias, int split,
                                         int co_lane, int wp, int g, int l16, int oh0, int ow0, bool with_bias = true)
    {
        constexpr unsigned kFar = 1u << 30;
        plane_b = (unsigned)a.h_out * a.w_out * 4u;
        c_out = a.c_out;
        relu = a.to_part ? 0 : a.relu;
        const unsigned out_b = (unsigned)a.c_out * plane_b;
        ro = make_rsrc(a.to_part ? part + (size_t)split * (out_b / 4) : out, out_b);
        // Output rows and columns left from this tile's corner (wave-uniform);
        // image sizes below 2^23 (checked with the plan) make the 24-bit
        // multiplies exact.
        const int rows = a.h_out - oh0, cols = a.w_out - ow0;
        const unsigned obase = (unsigned)(oh0 * a.w_out + ow0) * 4u;
#pragma unroll
        for (int n = 0; n < C::NB; ++n) {
            const int p = (wp * C::NB + n) * 16 + l16;
            const int q = p / C::TW, r = p - q * C::TW;
            const bool ok = p < C::NPIX && q < rows && r < cols;
            pix_off[n] = ok ? obase + (unsigned)(__mul24(q, a.w_out) + r) * 4u : kFar;
        }
#pragma unroll
        for (int m = 0; m < C::MA; ++m) {
            const int co = co_lane + 16 * m;
            chan_off[m] = co < a.c_out ? (unsigned)co * plane_b : kFar;
        }
        if (with_bias) load_bias(a, bias, co_lane, split);
        if constexpr (C::TAIL4) {
            // co_lane = co_base + 4*g; the tail uses co_base + 4*cg, cg = l16/4.
            tail_co = co_lane - 4 * g + 4 * (l16 >> 2);
            const int j = l16 & 3;
            const int p = (C::NB - 1) * 16 + j;
            const int q = p / C::TW, r = p - q * C::TW;
            const bool lane_stores = g == 0 && j < C::TAILP && q < rows && r < cols;
            tail_pix = lane_stores ? obase + (unsigned)(__mul24(q, a.w_out) + r) * 4u : kFar;
        }
    }

    // POOL: address the LDS tile instead of the output (after init): pixel p
    // of the tile at byte 4*p, channel co0 + c at byte 4*c*NPIX; pixels
    // outside the image or the tile and channels past C_out keep the
    // out-of-range offset and are not written.
    __device__ __forceinline__ void pool_init(float *tile, float *out, int co0, int co_lane, int wp, int g, int l16,
                                              int oh0, int ow0, const IgArgs &a)
    {
        constexpr unsigned kFar = 1u << 30;
        pl = tile;
        pool_co0 = co0;
        plane_b = 4u * C::NPIX;
        pool_hp = a.h_out / 2;
        pool_wpo = a.w_out / 2;
        pool_pi0 = oh0 / 2;
        pool_pj0 = ow0 / 2;
        pool_wc0 = co_lane - 4 * g - co0;
        pro = make_rsrc(out, (unsigned)a.c_out * (unsigned)pool_hp * (unsigned)pool_wpo * 4u);
        const int rows = a.h_out - oh0, cols = a.w_out - ow0;
#pragma unroll
        for (int n = 0; n < C::NB; ++n) {
            const int p = (wp * C::NB + n) * 16 + l16;
            const int q = p / C::TW, r = p - q * C::TW;
            const bool ok = p < C::NPIX && q < rows && r < cols;
            pix_off[n] = ok ? 4u * p : kFar;
        }
#pragma unroll
        for (int m = 0; m < C::MA; ++m) {
            const int co = co_lane + 16 * m;
            chan_off[m] = co < a.c_out ? 4u * (co - co0) * C::NPIX : kFar;
        }
        if constexpr (C::TAIL4) {
            const int j = l16 & 3;
            const int p = (C::NB - 1) * 16 + j;
            const int q = p / C::TW, r = p - q * C::TW;
            const bool lane_stores = g == 0 && j < C::TAILP && q < rows && r < cols;
            tail_pix = lane_stores ? 4u * p : kFar;
        }
    }

    // STREAM_POOL: pooled row i of this wave's 16*MA channels (tile rows 2i
    // and 2i + 1), read from the wave's own rows of the LDS tile, which this
    // wave wrote (LDS instructions of one wave complete in order).  Maxima
    // in the order pool_tile_finish takes them; windows with a pixel outside
    // the image have no output (floor) and channels past C_out none.
    __device__ __forceinline__ void pool_row(int i) const
    {
        constexpr int PWo = C::TW / 2, kOut = 16 * C::MA * PWo;
        const int lane = __lane_id();
        const int pi = pool_pi0 + i;
#pragma unroll
        for (int e0 = 0; e0 < kOut; e0 += 64) {
            const int e = e0 + lane;
            const int c = e / PWo, j = e - (e / PWo) * PWo;
            const int tc = pool_wc0 + c, co = pool_co0 + tc, pj = pool_pj0 + j;
            if (e < kOut && co < c_out && pi < pool_hp && pj < pool_wpo) {
                const float2 top = *reinterpret_cast<const float2 *>(pl + tc * C::NPIX + 2 * i * C::TW + 2 * j);
                const float2 bot = *reinterpret_cast<const float2 *>(pl + tc * C::NPIX + (2 * i + 1) * C::TW + 2 * j);
                float m = top.x, v = top.y;
                m = v > m ? v : m;
                v = bot.x;
                m = v > m ? v : m;
                v = bot.y;
                m = v > m ? v : m;
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, m), pro,
                                                      (int)((unsigned)((co * pool_hp + pi) * pool_wpo + pj) * 4u), 0,
                                                      C::SPOL);
            }
        }
    }

    // Row r of 16x16 block (m, n); the accumulator includes the bias.  Row r
    // is channel + r: r planes go into the scalar offset, so the four rows
    // share one vector offset.  A channel at or past C_out lies at or past
    // the descriptor's end (C_out planes), so its store is dropped.
    template <int RELU = 0>
    __device__ __forceinline__ void store_one(int m, int n, int r, float v) const
    {
        if constexpr (C::POOL) {
            constexpr unsigned kFar = 1u << 30;
            if ((chan_off[m] | pix_off[n]) < kFar) pl[(chan_off[m] + pix_off[n]) / 4 + r * C::NPIX] = fin<RELU>(v);
        } else {
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, fin<RELU>(v)), ro,
                                                  (int)(chan_off[m] + pix_off[n]), (int)(r * plane_b), C::SPOL);
        }
    }

    // Row r of the 4x4x1 tail block of m-block m: sum the four k-slice
    // partials, lane l getting (v[l] + v[l^16]) + (v[l^32] + v[l^48]) for
    // the first 16 lanes; lane 4*cg + j stores the channels that lanes
    // 16*cg.. hold the bias of.
    template <int RELU = 0>
    __device__ __forceinline__ void store_tail_one(int m, int r, float v) const
    {
        constexpr unsigned kFar = 1u << 30;
        const int src = 16 * ((__lane_id() & 15) >> 2);
        float s = v + __shfl_xor(v, 16);
        s += __shfl_xor(s, 32);
        const float tb = __shfl(b[m][r], src);
        const int co = tail_co + 16 * m + r;
        if constexpr (C::POOL) {
            if (co < c_out && tail_pix < kFar) pl[(co - pool_co0) * C::NPIX + tail_pix / 4] = fin<RELU>(s + tb);
        } else {
            const unsigned off = (co < c_out && tail_pix < kFar) ? (unsigned)co * plane_b + tail_pix : kFar;
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, fin<RELU>(s + tb)), ro, (int)off, 0,
                                                  C::SPOL);
        }
    }

    __device__ __forceinline__ void store(int m, int n, const floatx4 &v) const
    {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            if (C::TAIL4 && n == C::NB - 1) store_tail_one(m, r, v[r]);
            else store_one(m, n, r, v[r]);
        }
    }
};

// STREAM_POOL: the group iteration of compute_stage_streamed after which
// pooled row i (tile pixels up to (2i + 2)*TW - 1 in tile order) is all in
// LDS.  Group g's stores go out during iteration g + 1 (the last group's
// after the loop, "iteration kGroups"); the tail block's with group 0's.
template <class C>
constexpr int pool_row_ready(int i)
{
    const int last_px = (2 * i + 2) * C::TW - 1;
    const int last_full = 16 * C::NBM - 1;
    const int px = last_px < last_full ? last_px : last_full;
    return px / 16 / C::SGB + 1;
}

// The last stage of a one-channel-group-per-wave plan (NWK = 1), computed in
// groups of pixel blocks (Cfg::SGB, one block) with every step of the stage
// before moving to the next group, so that the output write overlaps the
// matrix work instead of following it: a finished group's stores are issued
// a few per step during the next group's steps, behind the step's matrix
// instructions.  (Issued in one burst they stall the wave, since every
// workgroup reaches the same group at about the same time and the burst is
// write bound.)  Smaller groups start the stores earlier and leave fewer
// after the last matrix instruction; a one-block group's chain of dependent
// 16x16x4 instructions still issues at the matrix pipe's rate.  Measured on
// 14x14 tiles (12 blocks + tail): groups of 1, 2, 3, 4, 6 and 12 blocks took
// 29.2, 29.5, 29.9, 30.4, 31.3 and 34.7 us with device-scope output stores,
// groups of 1 and 3 took 30.1 and 30.3 us with ordinary ones.  The 4x4x1
// tail block, if any, follows group 0 as one burst on its four accumulators
// and is stored with group 0.
template <class C, int RELU>
__device__ __forceinline__ void compute_stage_streamed(const float *xl, const AStage<C> &A,
                                                       const int (&b_base)[C::NB], floatx4 (&acc)[C::MA][C::NACC],
                                                       const Epilogue<C> &ep)
{
    constexpr int kSteps = C::KK * C::G4;
    constexpr int GB = C::SGB;
    constexpr int kGroups = (C::NBM + GB - 1) / GB;  // 16x16x4 groups
    static_assert(!C::TAIL4 || kGroups > 0, "the tail burst follows group 0");
    // Stores of one group, and of the tail (stored with group 0).
    constexpr int kGroupStores = C::MA * GB * 4;
    constexpr int kTailStores = C::TAIL4 ? C::MA * 4 : 0;
    constexpr int kDeferred = kGroupStores + kTailStores;
    constexpr int kStoreRate = (kDeferred + kSteps - 1) / kSteps;
    // B reads run DS steps ahead: a step here has only GB matrix
    // instructions, too few to cover an LDS read issued one step before.
    constexpr int DS = 2;
    float bv[DS + 1][GB];
    float avs[C::WL ? C::MA : 1][C::WL ? C::G4 : 1][C::WL ? C::KK : 1];
    if constexpr (C::WL) load_stage_a<C>(xl, A, avs);
    // The tail block's B values, read alongside group 0's (one more LDS read
    // per step) so that its instructions run back to back: a group of its
    // own would wait on an LDS read every ~10-cycle instruction.
    float tb[C::TAIL4 ? kSteps : 1];
    // Group grp covers blocks [grp*GB, min(grp*GB + GB, NBM)).
    auto read = [&](int grp, int st, float(&dst)[GB]) {
        const int t = st / C::G4, c4 = st % C::G4;
        const int kh = t / C::KS, kw = t % C::KS;
        const int off = C::CSTEP * c4 * C::PL + kh * C::HCP + kw;
#pragma unroll
        for (int j = 0; j < GB; ++j) {
            const int n = grp * GB + j;
            if (n < C::NBM) dst[j] = xl[b_base[n] + off];
        }
        if (C::TAIL4 && grp == 0) tb[st] = xl[b_base[C::NB - 1] + off];
    };
    // Store i of group grp (rows of its blocks, then, for group 0, the tail's).
    auto store_item = [&](int grp, int i) {
        if (i < kGroupStores) {
            const int m = i / (GB * 4), j = (i / 4) % GB, r = i % 4;
            const int n = grp * GB + j;
            if (n < C::NBM) ep.template store_one<RELU>(m, n, r, acc[m][n][r]);
        } else if (C::TAIL4 && grp == 0 && i < kDeferred) {
            const int m = (i - kGroupStores) / 4, r = (i - kGroupStores) % 4;
            ep.template store_tail_one<RELU>(m, r, acc[m][C::NB - 1][r]);
        }
    };
#pragma unroll
    for (int i = 0; i < DS && i < kGroups * kSteps; ++i) read(i / kSteps, i % kSteps, bv[i]);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int grp = 0; grp < kGroups; ++grp) {
#pragma unroll
        for (int st = 0; st < kSteps; ++st) {
            const int t = st / C::G4, c4 = st % C::G4;
            const int lin = grp * kSteps + st, cur = lin % (DS + 1), ahead = lin + DS;
            if (ahead < kGroups * kSteps) read(ahead / kSteps, ahead % kSteps, bv[ahead % (DS + 1)]);
#pragma unroll
            for (int m = 0; m < C::MA; ++m)
#pragma unroll
                for (int j = 0; j < GB; ++j) {
                    const int n = grp * GB + j;
                    if (n < C::NBM) {
                        float a_op;
                        if constexpr (C::WL) a_op = avs[m][c4][t];
                        else a_op = A.v[m][c4][t];
                        acc[m][n] = __builtin_amdgcn_mfma_f32_16x16x4f32(a_op, bv[cur][j], acc[m][n], 0, 0, 0);
                    }
                }
            if (grp > 0) {
#pragma unroll
                for (int k = 0; k < kStoreRate; ++k) store_item(grp - 1, st * kStoreRate + k);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        if constexpr (C::STREAM_POOL) {
            // Rows whose pixels are all in LDS now: group grp - 1's stores
            // went out during this group's steps.
            if (grp >= 1) {
                __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
                __builtin_amdgcn_wave_barrier();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
                for (int i = 0; i < C::TH / 2; ++i)
                    if (pool_row_ready<C>(i) == grp) ep.pool_row(i);
            }
        }
        if (C::TAIL4 && grp == 0) {
#pragma unroll
            for (int st = 0; st < kSteps; ++st) {
                const int t = st / C::G4, c4 = st % C::G4;
#pragma unroll
                for (int m = 0; m < C::MA; ++m) {
                    float a_op;
                    if constexpr (C::WL) a_op = avs[m][c4][t];
                    else a_op = A.v[m][c4][t];
                    acc[m][C::NB - 1 + st % 4] =
                        __builtin_amdgcn_mfma_f32_4x4x1f32(a_op, tb[st], acc[m][C::NB - 1 + st % 4], 0, 0, 0);
                }
            }
            fold_tail<C>(acc);
            __builtin_amdgcn_sched_barrier(0);
        }
    }
    // The last group's stores (and, with a single group, the tail's).
#pragma unroll
    for (int i = 0; i < kDeferred; ++i) store_item(kGroups - 1, i);
    if constexpr (C::STREAM_POOL) {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int i = 0; i < C::TH / 2; ++i)
            if (pool_row_ready<C>(i) == kGroups) ep.pool_row(i);
    }
}

// LDS writes of this wave done, then every wave: a bare barrier (the global
// stores in flight need not complete, and __syncthreads() would wait for
// them).  The empty asm statements keep the compiler from moving memory
// accesses across.
__device__ __forceinline__ void lds_barrier()
{
    __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt left at their maxima
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// The last stage streamed with the input channels split over waves
// (Cfg::SSPLIT): as compute_stage_streamed, group by group, but after each
// group (for group 0 with the tail burst, folded) the waves wk > 0 park the
// group's partial accumulators in `park` (double-buffered by group), one
// barrier, and the waves wk = 0 add them in wk order -- the order and sums
// of the unstreamed cross-wave sum, so the results are the same bits -- and
// store the group's outputs a few per step during the next group.  A
// group's park slot is written again two groups later, after the barrier
// that the readers reach only once they have read it.
template <class C, int RELU>
__device__ __forceinline__ void compute_stage_streamed_split(const float *xl, const AStage<C> &A,
                                                             const int (&b_base)[C::NB],
                                                             floatx4 (&acc)[C::MA][C::NACC], float *park, int wave,
                                                             int wk, int lane, const Epilogue<C> &ep)
{
    constexpr int kSteps = C::KK * C::G4;
    constexpr int GB = C::SGB;
    constexpr int kGroups = (C::NBM + GB - 1) / GB;
    constexpr int kGroupStores = C::MA * GB * 4;
    constexpr int kTailStores = C::TAIL4 ? C::MA * 4 : 0;
    constexpr int kDeferred = kGroupStores + kTailStores;
    constexpr int kStoreRate = (kDeferred + kSteps - 1) / kSteps;
    constexpr int DS = 2;
    constexpr int kWaveSlots = C::MA * C::SSLOTS * 4 * 64;  // floats per wave and group
    constexpr int kWaves = C::NWC * C::NWP;
    const int wcp = wave % kWaves;
    float bv[DS + 1][GB];
    float avs[C::WL ? C::MA : 1][C::WL ? C::G4 : 1][C::WL ? C::KK : 1];
    if constexpr (C::WL) load_stage_a<C>(xl, A, avs);
    float tb[C::TAIL4 ? kSteps : 1];
    auto read = [&](int grp, int st, float(&dst)[GB]) {
        const int t = st / C::G4, c4 = st % C::G4;
        const int kh = t / C::KS, kw = t % C::KS;
        const int off = C::CSTEP * c4 * C::PL + kh * C::HCP + kw;
#pragma unroll
        for (int j = 0; j < GB; ++j) {
            const int n = grp * GB + j;
            if (n < C::NBM) dst[j] = xl[b_base[n] + off];
        }
        if (C::TAIL4 && grp == 0) tb[st] = xl[b_base[C::NB - 1] + off];
    };
    auto store_item = [&](int grp, int i) {
        if (i < kGroupStores) {
            const int m = i / (GB * 4), j = (i / 4) % GB, r = i % 4;
            const int n = grp * GB + j;
            if (n < C::NBM) ep.template store_one<RELU>(m, n, r, acc[m][n][r]);
        } else if (C::TAIL4 && grp == 0 && i < kDeferred) {
            const int m = (i - kGroupStores) / 4, r = (i - kGroupStores) % 4;
            ep.template store_tail_one<RELU>(m, r, acc[m][C::NB - 1][r]);
        }
    };
    // Block slot j of group grp (j = GB: the tail, group 0 only).
    auto block_of = [&](int grp, int j) { return j < GB ? grp * GB + j : C::NB - 1; };
    auto slot_used = [&](int grp, int j) {
        return j < GB ? grp * GB + j < C::NBM : (C::TAIL4 && grp == 0);
    };
    auto sum_group = [&](int grp) {
        float *const buf = park + (grp & 1) * (C::NWK - 1) * kWaves * kWaveSlots;
        if (wk > 0) {
            float *dst = buf + ((wk - 1) * kWaves + wcp) * kWaveSlots + lane;
#pragma unroll
            for (int m = 0; m < C::MA; ++m)
#pragma unroll
                for (int j = 0; j < C::SSLOTS; ++j)
                    if (slot_used(grp, j)) {
#pragma unroll
                        for (int r = 0; r < 4; ++r) dst[((m * C::SSLOTS + j) * 4 + r) * 64] = acc[m][block_of(grp, j)][r];
                    }
        }
        lds_barrier();
        if (wk == 0) {
#pragma unroll
            for (int k = 1; k < C::NWK; ++k) {
                const float *src = buf + ((k - 1) * kWaves + wcp) * kWaveSlots + lane;
#pragma unroll
                for (int m = 0; m < C::MA; ++m)
#pragma unroll
                    for (int j = 0; j < C::SSLOTS; ++j)
                        if (slot_used(grp, j)) {
#pragma unroll
                            for (int r = 0; r < 4; ++r)
                                acc[m][block_of(grp, j)][r] += src[((m * C::SSLOTS + j) * 4 + r) * 64];
                        }
            }
        }
    };
#pragma unroll
    for (int i = 0; i < DS && i < kGroups * kSteps; ++i) read(i / kSteps, i % kSteps, bv[i]);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int grp = 0; grp < kGroups; ++grp) {
#pragma unroll
        for (int st = 0; st < kSteps; ++st) {
            const int t = st / C::G4, c4 = st % C::G4;
            const int lin = grp * kSteps + st, cur = lin % (DS + 1), ahead = lin + DS;
            if (ahead < kGroups * kSteps) read(ahead / kSteps, ahead % kSteps, bv[ahead % (DS + 1)]);
#pragma unroll
            for (int m = 0; m < C::MA; ++m)
#pragma unroll
                for (int j = 0; j < GB; ++j) {
                    const int n = grp * GB + j;
                    if (n < C::NBM) {
                        float a_op;
                        if constexpr (C::WL) a_op = avs[m][c4][t];
                        else a_op = A.v[m][c4][t];
                        acc[m][n] = __builtin_amdgcn_mfma_f32_16x16x4f32(a_op, bv[cur][j], acc[m][n], 0, 0, 0);
                    }
                }
            if (grp > 0 && wk == 0) {
#pragma unroll
                for (int k = 0; k < kStoreRate; ++k) store_item(grp - 1, st * kStoreRate + k);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        if (C::TAIL4 && grp == 0) {
#pragma unroll
            for (int st = 0; st < kSteps; ++st) {
                const int t = st / C::G4, c4 = st % C::G4;
#pragma unroll
                for (int m = 0; m < C::MA; ++m) {
                    float a_op;
                    if constexpr (C::WL) a_op = avs[m][c4][t];
                    else a_op = A.v[m][c4][t];
                    acc[m][C::NB - 1 + st % 4] =
                        __builtin_amdgcn_mfma_f32_4x4x1f32(a_op, tb[st], acc[m][C::NB - 1 + st % 4], 0, 0, 0);
                }
            }
            fold_tail<C>(acc);
        }
        sum_group(grp);
        __builtin_amdgcn_sched_barrier(0);
    }
    if (wk == 0) {
#pragma unroll
        for (int i = 0; i < kDeferred; ++i) store_item(kGroups - 1, i);
    }
}

// The last stage and the output.  NWK = 1: streamed.  NWK > 1: compute, then
// sum the NWK channel-group partials (waves wk > 0 park theirs in LDS once
// every wave is past the last stage, waves wk = 0 add and store).
template <class C>
__device__ __forceinline__ void final_stage(const float *xl, const AStage<C> &A, const int (&b_base)[C::NB],
                                            floatx4 (&acc)[C::MA][C::NACC], float *park_area, int wave, int wk,
                                            int lane, const Epilogue<C> &ep)
{
    if constexpr (C::NWK == 1 && (!C::POOL || C::STREAM_POOL)) {
        // The ReLU choice is made once here: per store it cost a compare, a
        // mask and a select (with their register hazards) between the
        // matrix instructions.  STREAM_POOL: the stores go to the LDS tile
        // and the wave pools its rows as they fill.
        if (ep.relu) compute_stage_streamed<C, 2>(xl, A, b_base, acc, ep);
        else compute_stage_streamed<C, 1>(xl, A, b_base, acc, ep);
    } else if constexpr (C::SSPLIT && !C::POOL) {
        // park_area is the streamed split's own LDS area here (Cfg::PARKS).
        if (ep.relu) compute_stage_streamed_split<C, 2>(xl, A, b_base, acc, park_area, wave, wk, lane, ep);
        else compute_stage_streamed_split<C, 1>(xl, A, b_base, acc, park_area, wave, wk, lane, ep);
    } else if constexpr (C::NWK == 1) {
        // PoolTile with pixels split over waves: the results go to LDS,
        // whose queue the matrix steps' operand reads use; written in one
        // burst after the stage instead of between its steps, and pooled
        // by the workgroup (pool_tile_finish) after a barrier.
        NoNextStage none;
        compute_stage<C>(xl, A, b_base, acc, none);
        fold_tail<C>(acc);
#pragma unroll
        for (int m = 0; m < C::MA; ++m)
#pragma unroll
            for (int n = 0; n < C::NB; ++n) ep.store(m, n, acc[m][n]);
    } else {
        NoNextStage none;
        compute_stage<C>(xl, A, b_base, acc, none);
        fold_tail<C>(acc);
        __syncthreads();
        constexpr int per_wave = C::MA * C::NB * 4 * 64;
        const int wcp = wave % (C::NWC * C::NWP);
        if (wk > 0) {
            float *park = park_area + ((wk - 1) * C::NWC * C::NWP + wcp) * per_wave + lane;
#pragma unroll
            for (int m = 0; m < C::MA; ++m)
#pragma unroll
                for (int n = 0; n < C::NB; ++n)
#pragma unroll
                    for (int r = 0; r < 4; ++r) park[((m * C::NB + n) * 4 + r) * 64] = acc[m][n][r];
        }
        __syncthreads();
        if (wk > 0) return;
#pragma unroll
        for (int k = 1; k < C::NWK; ++k) {
            const float *src = park_area + ((k - 1) * C::NWC * C::NWP + wcp) * per_wave + lane;
#pragma unroll
            for (int m = 0; m < C::MA; ++m)
#pragma unroll
                for (int n = 0; n < C::NB; ++n)
#pragma unroll
                    for (int r = 0; r < 4; ++r) acc[m][n][r] += src[((m * C::NB + n) * 4 + r) * 64];
        }
#pragma unroll
        for (int m = 0; m < C::MA; ++m)
#pragma unroll
            for (int n = 0; n < C::NB; ++n) ep.store(m, n, acc[m][n]);
    }
}

// The fewest loads any wave issues for one stage: its full rounds of halo
// DMA (a last, partial round falls to some waves only) and its weight loads.
template <class C, class WS>
constexpr int kStageLoads()
{
    return NextStage<C, WS>::kFull + WS::NA_MIN;
}

// Loads a wave may leave in flight at the end of stage s (those of stages
// s + 2 .. s + NBUF - 1 that exist) while stage s + 1's have all landed.
template <class C, class WS>
constexpr int kKeepAfter(int s)
{
    const int last = s + C::NBUF - 1 < C::NS - 1 ? s + C::NBUF - 1 : C::NS - 1;
    const int n = last - (s + 2) + 1;
    return n > 0 ? n * kStageLoads<C, WS>() : 0;
}

// The stages of a fixed-stage plan, unrolled at compile time: stage s
// computes from buffer s mod NBUF and issues the loads of stage s + NBUF - 1
// (into the buffer stage s - 1 read, which every wave finished before the
// barrier that ended it), and the last stage is the final one.  Every wait
// is exact: it leaves in flight only the loads of the stages after next.
template <class C, class WS, int... S>
__device__ __forceinline__ void run_stages(std::integer_sequence<int, S...>, float *const (&bufs)[6],
                                           AStage<C> *const (&regs)[6], const float *__restrict__ x,
                                           const IgArgs &a, const WeightCtx &wctx, int c_begin, int wave, int wk,
                                           int lane, const int (&xo)[C::XPT], const int (&b_base)[C::NB],
                                           floatx4 (&acc)[C::MA][C::NACC], const Epilogue<C> &ep)
{
    auto stage = [&](auto sc) {
        constexpr int s = decltype(sc)::value;
        constexpr int t = s + C::NBUF - 1;  // the stage whose loads this one issues
        constexpr int keep = kKeepAfter<C, WS>(s);
        float *xl = bufs[s % C::NBUF];
        AStage<C> &A = *regs[s % C::NBUF];
        if constexpr (s == C::NS - 1) {
            final_stage<C>(xl, A, b_base, acc, bufs[0], wave, wk, lane, ep);
        } else {
            if constexpr (t < C::NS) {
                NextStage<C, WS> next(bufs[t % C::NBUF], *regs[t % C::NBUF], x, a, wctx, (c_begin + t) * C::CC, wave,
                                      xo);
                compute_stage<C>(xl, A, b_base, acc, next);
            } else {
                NoNextStage none;
                compute_stage<C>(xl, A, b_base, acc, none);
            }
            stage_wait<C, keep>();
        }
    };
    for_each_index(std::integer_sequence<int, S...>{}, stage);
}

// The stages of a two-buffer plan from stage ch (in bA / rA, landed) on:
// stage s computes from one buffer while the loads of stage s + 1 fill the
// other, then waits for them; the last stage is the final one.
template <class C, class WS>
__device__ __forceinline__ void stage_loop(float *bA, AStage<C> &rA, float *bB, AStage<C> &rB, float *park, int ch,
                                           int c_end, const float *__restrict__ x, const IgArgs &a,
                                           const WeightCtx &wctx, int wave, int wk, int lane,
                                           const int (&xo)[C::XPT], const int (&b_base)[C::NB],
                                           floatx4 (&acc)[C::MA][C::NACC], const Epilogue<C> &ep)
{
    for (;; ch += 2) {
        if (ch + 1 >= c_end) {
            final_stage<C>(bA, rA, b_base, acc, park, wave, wk, lane, ep);
            break;
        }
        {
            NextStage<C, WS> next(bB, rB, x, a, wctx, (ch + 1) * C::CC, wave, xo);
            compute_stage<C>(bA, rA, b_base, acc, next);
        }
        stage_ready();
        if (ch + 2 >= c_end) {
            final_stage<C>(bB, rB, b_base, acc, park, wave, wk, lane, ep);
            break;
        }
        {
            NextStage<C, WS> next(bA, rA, x, a, wctx, (ch + 2) * C::CC, wave, xo);
            compute_stage<C>(bB, rB, b_base, acc, next);
        }
        stage_ready();
    }
}

// Arrivals per output tile for the fused split sum.  Zero when the module
// loads; the workgroup that completes a tile puts its count back to zero, so
// the array is zero again whenever no call is running.
constexpr int kMaxFusedTiles = 1 << 16;
// The fused split sum is used when each thread of the finishing workgroup
// loads at most kFuseMaxLoads partial sums (outputs per thread x splits).
// Measured on MI355X: with one output of 4 slices per thread it saves the
// second launch (1x1 512->512 at 7x7: 6.86 -> 6.46 us per call); with 4
// outputs of 8 slices it costs more than it saves (5x5 at 7x7: 12.95 ->
// 14.58 us), and larger tiles leave the sum to sum_splits, which spreads it
// over the whole GPU instead of the tiles' last workgroups.
constexpr int kFuseElems = 4;  // outputs per thread and pass of the finishing loop
constexpr int kFuseMaxLoads = 8;
__device__ unsigned g_split_arrivals[kMaxFusedTiles];

// Fused split sum.  Every workgroup of a tile has stored its partial sums at
// device scope to slice `split` of `part`; once those stores have completed it
// counts itself in, and the last of the tile's `splits` workgroups adds the
// slices in split order (the order and arithmetic of sum_splits, so the
// values do not depend on which workgroup is last), applies ReLU and writes
// the tile's outputs.  Its loads are device-scope loads, which see the other
// workgroups' stores however the XCDs' L2 caches hold them.
//
// Why the order holds without a release/acquire fence pair.  In the AMDGPU
// backend's memory model for this GPU family (LLVM's AMDGPUUsage, "Memory
// Model GFX942", which covers gfx950), agent-scope atomic stores, loads and
// read-modify-writes are ordinary memory instructions with the SC1 cache
// policy: they are performed at the level the XCDs share (each XCD's L2 is
// not coherent with the others; SC1 writes through it and SC1 loads do not
// take a stale line from it).  A release at agent scope is "write back the
// L2 (buffer_wbl2 sc1), then s_waitcnt vmcnt(0)", and an acquire is
// "s_waitcnt vmcnt(0), then invalidate the L2 (buffer_inv sc1)"; the L2
// write-back and invalidate exist only for data that ordinary (non-SC1)
// accesses leave in or take from an XCD's L2.  Here every access to `part`
// on this path is SC1, so:
//  * writer side: the partial sums are SC1 stores; s_waitcnt vmcnt(0) waits
//    until each has been acknowledged by the shared level; only then does the
//    barrier let thread 0 issue the arrival count's atomic add.  That is the
//    release sequence without the write-back, which SC1 stores do not need.
//  * reader side: thread 0 of the last workgroup receives the atomic's
//    result (the wait for it is a data dependency), publishes it through LDS
//    and a barrier, and only then do the SC1 loads of the slices issue, which
//    read the shared level.  That is the acquire sequence without the L2
//    invalidate, which SC1 loads do not need.
// A device-scope __threadfence() on both sides (the write-back and
// invalidate of whole L2 caches) was measured at +45 to +60 us per call.
__device__ __forceinline__ float load_device_scope(const float *p)
{
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <class C>
__device__ __forceinline__ void finish_split_tile(const IgArgs &a, const float *part, float *out, int tile, int co0,
                                                  int oh0, int ow0, unsigned *last_lds)
{
    __builtin_amdgcn_s_waitcnt(0);  // this thread's partial-sum stores have completed
    __syncthreads();
    if (threadIdx.x == 0) {
        const unsigned prev = atomicAdd(&g_split_arrivals[tile], 1u);
        const unsigned last = prev + 1 == (unsigned)a.splits ? 1u : 0u;
        if (last) atomicExch(&g_split_arrivals[tile], 0u);
        *last_lds = last;
    }
    __syncthreads();
    if (*last_lds == 0u) return;
    // Up to kFuseElems outputs per thread and pass, with the loads of all
    // their slices (kB at a time) in flight before any is added: a pass costs
    // about one round trip to the shared cache level.
    constexpr int kTP = C::TH * C::TW;
    constexpr int kB = 8;
    const int64_t slice = (int64_t)a.c_out * a.h_out * a.w_out;
    // The output is below 2^30 bytes (checked when the plan is made).
    const __amdgpu_buffer_rsrc_t ro = make_rsrc(out, (unsigned)slice * 4u);
    for (int e0 = threadIdx.x; e0 < C::COT * kTP; e0 += kFuseElems * C::NT) {
        int64_t off[kFuseElems];
        bool ok[kFuseElems];
        float v[kFuseElems];
#pragma unroll
        for (int j = 0; j < kFuseElems; ++j) {
            const int e = e0 + j * C::NT;
            const int c = e / kTP;
            const int p = e - c * kTP;
            const int q = p / C::TW;
            const int oh = oh0 + q, ow = ow0 + (p - q * C::TW), co = co0 + c;
            ok[j] = e < C::COT * kTP && co < a.c_out && oh < a.h_out && ow < a.w_out;
            off[j] = ok[j] ? ((int64_t)co * a.h_out + oh) * a.w_out + ow : 0;
            v[j] = ok[j] ? load_device_scope(part + off[j]) : 0.f;
        }
        for (int k = 1; k < a.splits; k += kB) {
            float t[kFuseElems][kB];
#pragma unroll
            for (int j = 0; j < kFuseElems; ++j)
#pragma unroll
                for (int b = 0; b < kB; ++b)
                    if (ok[j] && k + b < a.splits) t[j][b] = load_device_scope(part + off[j] + (k + b) * slice);
#pragma unroll
            for (int j = 0; j < kFuseElems; ++j)
#pragma unroll
                for (int b = 0; b < kB; ++b)
                    if (ok[j] && k + b < a.splits) v[j] += t[j][b];
        }
#pragma unroll
        for (int j = 0; j < kFuseElems; ++j)
            if (ok[j]) {
                const float r = a.relu && v[j] < 0.f ? 0.f : v[j];
                if constexpr (C::OPOL != 0)
                    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, r), ro, (int)(off[j] * 4), 0,
                                                          C::OPOL);
                else
                    out[off[j]] = r;
            }
    }
}

// PoolTile: every wave has written its results to the LDS tile; each output
// of the pooled tile is the maximum of its 2x2 window, compared in the order
// (0,0), (0,1), (1,0), (1,1) as the pool kernels do.  Windows lie inside the
// tile (even sides, tiles start at even coordinates); a window with any pixel
// outside the image has no pooled output (floor), and channels past C_out
// are not written.
template <class C>
__device__ __forceinline__ void pool_tile_finish(const float *tile, float *out, const IgArgs &a, int co0, int oh0,
                                                 int ow0)
{
    __syncthreads();
    constexpr int PH = C::TH / 2, PW = C::TW / 2;
    const int hp = a.h_out / 2, wpo = a.w_out / 2;
    const int pi0 = oh0 / 2, pj0 = ow0 / 2;
    // With a cache policy on the output (SC1), the stores carry it as the
    // full-size stores do; the pooled output is below 2^31 bytes (the plan
    // checks the full-size one).
    const __amdgpu_buffer_rsrc_t ro = make_rsrc(out, (unsigned)a.c_out * (unsigned)hp * (unsigned)wpo * 4u);
    for (int e = threadIdx.x; e < C::COT * PH * PW; e += C::NT) {
        const int c = e / (PH * PW);
        const int q = e - c * (PH * PW);
        const int i = q / PW, j = q - (q / PW) * PW;
        const int co = co0 + c, pi = pi0 + i, pj = pj0 + j;
        if (co >= a.c_out || pi >= hp || pj >= wpo) continue;
        // Even NPIX and TW: each window row is an aligned pair.
        const float2 top = *reinterpret_cast<const float2 *>(tile + c * C::NPIX + 2 * i * C::TW + 2 * j);
        const float2 bot = *reinterpret_cast<const float2 *>(tile + c * C::NPIX + (2 * i + 1) * C::TW + 2 * j);
        float m = top.x, v = top.y;
        m = v > m ? v : m;
        v = bot.x;
        m = v > m ? v : m;
        v = bot.y;
        m = v > m ? v : m;
        if constexpr (C::SPOL != 0)
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, m), ro,
                                                  (int)((unsigned)((co * hp + pi) * wpo + pj) * 4u), 0, C::SPOL);
        else
            out[((int64_t)co * hp + pi) * wpo + pj] = m;
    }
}

template <class C, bool PK>
__global__ __launch_bounds__(C::NT) void conv_igemm(const float *__restrict__ x, const float *__restrict__ w,
                                                    const float *__restrict__ bias, float *__restrict__ out,
                                                    float *__restrict__ part, IgArgs a)
{
    // Stage buffers in separate LDS objects, so the compiler can tell a read
    // of one from the DMA filling another.
    __shared__ __attribute__((aligned(16))) float lds0[C::BUF0];
    __shared__ __attribute__((aligned(16))) float lds1[C::SBUF];
    __shared__ __attribute__((aligned(16))) float lds2[C::NBUF > 2 ? C::SBUF : 1];
    __shared__ __attribute__((aligned(16))) float lds3[C::NBUF > 3 ? C::SBUF : 1];
    __shared__ __attribute__((aligned(16))) float lds4[C::NBUF > 4 ? C::SBUF : 1];
    __shared__ __attribute__((aligned(16))) float lds5[C::NBUF > 5 ? C::SBUF : 1];
    // The first stage's channel groups (PF).
    constexpr bool kPF = C::PF;
    __shared__ __attribute__((aligned(16))) float gb0[kPF ? C::GSZ : 1];
    __shared__ __attribute__((aligned(16))) float gb1[kPF ? C::GSZ : 1];
    __shared__ __attribute__((aligned(16))) float gb2[kPF && C::G4 > 2 ? C::GSZ : 1];
    __shared__ __attribute__((aligned(16))) float gb3[kPF && C::G4 > 3 ? C::GSZ : 1];
    __shared__ unsigned last_arrival[1];  // fused split sum: this workgroup completes its tile
    __shared__ __attribute__((aligned(16))) float pool_lds[C::POOL ? C::POOL_FLOATS : 1];  // PoolTile's tile
    constexpr bool kStreamSplit = C::SSPLIT && !C::POOL;
    __shared__ __attribute__((aligned(16))) float park_s[kStreamSplit ? C::PARKS : 1];  // streamed split sums

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    __builtin_assume(wave >= 0 && wave < C::NW);  // lets per-wave index arithmetic fold
    const int wc = wave % C::NWC;
    const int wp = (wave / C::NWC) % C::NWP;
    const int wk = wave / (C::NWC * C::NWP);
    const int g = lane >> 4;
    const int l16 = lane & 15;

    // Workgroup -> (split, tile).  Workgroups are dealt round-robin to the 8
    // XCDs (workgroup i to XCD i mod 8), each with its own L2; giving every
    // XCD a contiguous run of tiles keeps tiles that share data in one L2:
    // neighbouring spatial tiles (halo rows, output cache lines, and with
    // sp_fast the same weights) or, otherwise, the output-channel tiles of
    // one spatial tile (the same input).
    const int nwg = (int)gridDim.x;
    const int xcd = (int)blockIdx.x % 8, slot = (int)blockIdx.x / 8;
    const int per = nwg / 8, extra = nwg % 8;
    const int lin = xcd * per + min(xcd, extra) + slot;
    const int split = (int)fast_div((unsigned)lin, a.ntiles);
    const int tile = lin - split * (int)a.ntiles.d;
    int sp, co_t;
    if (a.sp_fast) {
        co_t = (int)fast_div((unsigned)tile, a.sp_tiles);
        sp = tile - co_t * (int)a.sp_tiles.d;
    } else {
        sp = (int)fast_div((unsigned)tile, a.co_tiles);
        co_t = tile - sp * (int)a.co_tiles.d;
    }
    const int th_i = (int)fast_div((unsigned)sp, a.tiles_w);
    const int tw_i = sp - th_i * (int)a.tiles_w.d;
    const int co0 = co_t * C::COT;
    const int oh0 = th_i * C::TH, ow0 = tw_i * C::TW;
    const int ih0 = oh0 * C::S - a.pad, iw0 = ow0 * C::S - a.pad;
    const int c_begin = split * a.chunks_per_split;
    const int c_end = min(c_begin + a.chunks_per_split, a.nchunks);

    // Weight operand: lane (g, l16) of m-block m holds output channel
    // co0 + wc*16*MA + 16*m + l16, from OIHW or from the prepacked layout.
    // (Weights through LDS read OIHW; a variant's prepacked weights are an
    // OIHW copy.)
    using WS = typename std::conditional<C::WL, LdsWeights<C>,
                                         typename std::conditional<PK, PackedWeights<C>, OihwWeights<C>>::type>::type;
    const int ci_lane = 4 * wk + g;
    WeightCtx wctx;
    wctx.rw = make_rsrc(w, PK ? a.co_tiles.d * (unsigned)a.nchunks * (C::COT * C::CC * C::KK * 4u)
                              : (unsigned)a.c_out * a.c_in * C::KK * 4u);
    wctx.c_in = a.c_in;
    wctx.nchunks = a.nchunks;
    wctx.co_lane0 = co0 + wc * 16 * C::MA + l16;
    wctx.ci_lane = ci_lane;
    wctx.block0 = (co_t * a.nchunks * C::NWK + wk) * C::NWC + wc;
    wctx.lane = lane;
    wctx.wave = wave;
    wctx.c_out = a.c_out;
    wctx.w = w;
    WlLanes<C> wl_lanes;
    if constexpr (C::WL) wl_lanes.init(co0, a.c_in, a.c_out, wave, lane);
    wctx.wl = &wl_lanes;

    // The first stage's loads go out before the rest of the set-up: with one
    // wave per SIMD every vector instruction of the set-up costs its full
    // issue time, so it runs while the loads are in flight.
    int xo[C::XPT];
    halo_offsets<C>(xo, a, wave, lane, ih0, iw0);
    AStage<C> a0, a1;
    if constexpr (C::WL) {
#pragma unroll
        for (int m = 0; m < C::MA; ++m)
            a0.base[m] = C::XSZ + (4 * wk + g) * C::CPL + (wc * 16 * C::MA + 16 * m + l16) * C::KKP;
        a1 = a0;
    }
    const WS ws0(wctx, a.c_out, c_begin * C::CC, lds0);
    Epilogue<C> ep;
    const __amdgpu_buffer_rsrc_t rx0 = halo_rsrc(x, a, c_begin * C::CC);
    if constexpr (kPF) {
        // The bias goes first, so that every load after it belongs to the
        // first stage or the next (their waits count exactly those); then
        // channel group 0's halo and weights.
        ep.load_bias(a, bias, co0 + wc * 16 * C::MA + 4 * g, split);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int i = 0; i < 4; ++i) dma_group<C>(gb0, rx0, 0, i, wave, xo);
#pragma unroll
        for (int q = 0; q <= WS::group_last(0); ++q) ws0.load(q, a0);
    } else {
        dma_halo<C>(lds0, rx0, wave, xo);
        load_a<C>(a0, ws0);
    }
    __builtin_amdgcn_sched_barrier(0);

    // Input operand: LDS base of each pixel block for this lane.
    int b_base[C::NB];
#pragma unroll
    for (int nb = 0; nb < C::NB; ++nb) {
        int p = (wp * C::NB + nb) * 16 + ((C::TAIL4 && nb == C::NB - 1) ? (l16 & 3) : l16);
        if (p >= C::NPIX) p = 0;  // padding lanes read a valid word; never stored
        b_base[nb] = ci_lane * C::LSTEP * C::PL + (p / C::TW) * C::S * C::HCP + (p % C::TW) * C::S;
    }

    // Output side, set up before the last stage so that its stores can stream
    // out while the last blocks are still being computed.  Accumulator block
    // (m, n), register r holds output channel co0 + wc*16*MA + 16*m + 4*g + r
    // at tile pixel (wp*NB + n)*16 + l16 (the 4x4x1 tail block is laid out
    // as its Cfg comment says).  With to_part, workgroups write slice `split`
    // of the partial sums, in the output's layout, without bias or ReLU.
    // Stores go through a buffer descriptor: a lane outside the output (pixel
    // or channel) gets an offset of at least 2^30 bytes, past the descriptor's
    // range (< 2^30, checked when the plan is made), and its store is dropped.
    ep.init(a, out, part, bias, split, co0 + wc * 16 * C::MA + 4 * g, wp, g, l16, oh0, ow0, !kPF);
    if constexpr (C::POOL) ep.pool_init(pool_lds, out, co0, co0 + wc * 16 * C::MA + 4 * g, wp, g, l16, oh0, ow0, a);

    // The 16x16x4 blocks' accumulators start from the bias (zero for splits
    // other than 0, and for the waves wk > 0 whose partials are added to wave
    // wk = 0's), so the stores need no addition; the 4x4x1 tail block's four k-slice
    // accumulators start from zero and get the bias when they are summed.
    floatx4 acc[C::MA][C::NACC];
#pragma unroll
    for (int m = 0; m < C::MA; ++m)
#pragma unroll
        for (int n = 0; n < C::NACC; ++n)
            acc[m][n] = (n < C::NBM && wk == 0) ? floatx4{ep.b[m][0], ep.b[m][1], ep.b[m][2], ep.b[m][3]}
                                                : floatx4{0.f, 0.f, 0.f, 0.f};

    if constexpr (C::NBUF > 2) {
        // A deeper pipeline: stages 1 .. NBUF - 2 are issued now, stage s
        // issues stage s + NBUF - 1 (see run_stages).
        AStage<C> ax[4];
        if constexpr (C::WL) ax[0] = ax[1] = ax[2] = ax[3] = a0;
        float *const bufs[6] = {lds0, lds1, lds2, lds3, lds4, lds5};
        AStage<C> *const regs[6] = {&a0, &a1, &ax[0], &ax[1], &ax[2], &ax[3]};
        constexpr int kAhead = C::NBUF - 2 < C::NS - 1 ? C::NBUF - 2 : C::NS - 1;  // stages issued here
        for_each_index(std::make_integer_sequence<int, kAhead>{}, [&](auto tc) {
            constexpr int t = decltype(tc)::value + 1;
            dma_halo<C>(bufs[t], halo_rsrc(x, a, (c_begin + t) * C::CC), wave, xo);
            load_a<C>(*regs[t], WS(wctx, a.c_out, (c_begin + t) * C::CC, bufs[t]));
        });
        stage_wait<C, kAhead * kStageLoads<C, WS>()>();
        run_stages<C, WS>(std::make_integer_sequence<int, C::NS>{}, bufs, regs, x, a, wctx, c_begin, wave, wk, lane,
                          xo, b_base, acc, ep);
        if constexpr (C::FUSED) finish_split_tile<C>(a, part, out, tile, co0, oh0, ow0, last_arrival);
        if constexpr (C::POOL && !C::STREAM_POOL) pool_tile_finish<C>(pool_lds, out, a, co0, oh0, ow0);
        return;
    }

    stage_ready();
    if constexpr (kPF) {
        // At least two stages (checked when the plan is made): the first
        // from the group buffers, the second from lds1, and so on.
        // Group c's buffer (c is a constant wherever this is called).
        auto gb = [&](int c) -> float * { return c == 0 ? gb0 : c == 1 ? gb1 : c == 2 ? gb2 : gb3; };
        {
            NextStage<C, WS> next(lds1, a1, x, a, wctx, (c_begin + 1) * C::CC, wave, xo);
            first_stage<C>(gb, rx0, ws0, a0, xo, wave, b_base, acc, next);
        }
        stage_ready();
        stage_loop<C, WS>(lds1, a1, lds0, a0, kStreamSplit ? park_s : lds0, c_begin + 1, c_end, x, a, wctx, wave,
                          wk, lane, xo, b_base, acc, ep);
    } else {
        stage_loop<C, WS>(lds0, a0, lds1, a1, kStreamSplit ? park_s : lds0, c_begin, c_end, x, a, wctx, wave, wk,
                          lane, xo, b_base, acc, ep);
    }
    if constexpr (C::FUSED) finish_split_tile<C>(a, part, out, tile, co0, oh0, ow0, last_arrival);
    if constexpr (C::POOL && !C::STREAM_POOL) pool_tile_finish<C>(pool_lds, out, a, co0, oh0, ow0);
}


template <class C>
void launch_cfg(dim3 grid, hipStream_t st, const float *x, const float *w, const float *b, float *o, float *ws,
                const IgArgs &a, bool packed)
{
    if constexpr (C::POOLABLE) {
        if (a.pool_tile) {
            if (packed) hipLaunchKernelGGL((conv_igemm<PoolTile<C>, true>), grid, dim3(C::NT), 0, st, x, w, b, o, ws, a);
            else hipLaunchKernelGGL((conv_igemm<PoolTile<C>, false>), grid, dim3(C::NT), 0, st, x, w, b, o, ws, a);
            return;
        }
    }
    using F = FusedSplit<C>;
    if (a.fuse) {
        if (packed) hipLaunchKernelGGL((conv_igemm<F, true>), grid, dim3(C::NT), 0, st, x, w, b, o, ws, a);
        else hipLaunchKernelGGL((conv_igemm<F, false>), grid, dim3(C::NT), 0, st, x, w, b, o, ws, a);
    } else if (a.to_part) {
        // (A configuration whose stores are at device scope already serves.)
        using P = typename std::conditional<C::SPOL == kPolicyDeviceScope, C, SplitPart<C>>::type;
        if (packed) hipLaunchKernelGGL((conv_igemm<P, true>), grid, dim3(C::NT), 0, st, x, w, b, o, ws, a);
        else hipLaunchKernelGGL((conv_igemm<P, false>), grid, dim3(C::NT), 0, st, x, w, b, o, ws, a);
    } else {
        if (packed) hipLaunchKernelGGL((conv_igemm<C, true>), grid, dim3(C::NT), 0, st, x, w, b, o, ws, a);
        else hipLaunchKernelGGL((conv_igemm<C, false>), grid, dim3(C::NT), 0, st, x, w, b, o, ws, a);
    }
}

template <class C>
constexpr Variant make_variant(const char *name)
{
    return Variant{name, C::KS, C::S, C::TH, C::TW, C::NWC, C::NWP, C::NWK, C::MA, C::CC,
                   C::NT, C::COT, C::LDS_BYTES, C::NS, C::WL, C::NBUF, C::PF, C::POOLABLE, C::C1,
                   &launch_cfg<C>};
}

}  // namespace
}  // namespace ilpm
