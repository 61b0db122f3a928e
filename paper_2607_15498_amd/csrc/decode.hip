// Rank-space decode attention over the compressed cache, gfx950.
//
// Attention over the reconstructed cache of Eq. (6) without reconstructing it: with an
// orthonormal key basis <q, P_K^T (m . c)> = <P_K q, m . c>, and the value side is linear,
// so  o = P_V^T (sum_t p_t m_t . c^V_t) + sum_e p_e v_e.
//
// Grid: (n_wg + 1) workgroups per unit (sequence, KV head, tile of up to 16 query rows,
// row = query * H/G + head), on a 1D grid in which consecutive workgroups take consecutive
// units.  Workgroup x = 0 attends to the exact slots (window + appended tokens) in the
// original space; workgroup x >= 1 streams the 16-token tiles [(x-1) tpw, x tpw) of KV head
// g's stored tokens (tile t = chunk t/16, slots 16 (t%16)..).  Per workgroup (8 waves, two
// workgroups per CU):
//   1. the chunks' stored ranks are fetched with one vector load per 16 tokens and turned
//      into tile offsets; q' = P_K[g] q / sqrt(d) by MFMA (basis split into bf16 hi + lo
//      parts, ~2^-16 error);
//   2. the tile range is cut into rounds that fit one 16 KB buffer per stream; two rounds
//      are in flight at a time (double-buffered direct-to-LDS loads, a fixed number per
//      wave and round), so a round's tiles run while the next round lands;
//   3. waves take 16-token tiles of the rank-sorted storage and gather their MFMA operands
//      from the tile rectangles in LDS: 16-byte row pieces for the score tile (16 tokens x
//      32 coefficients per step) and, for the value tile, 4 positions at one coordinate.
//      The score C fragment (lane = query row, 4 tokens) is the B operand of the transposed
//      16x16x16 value MFMA, so the online softmax is lane-local;
//   4. the waves' (max, sum, acc) are combined in a fixed order into one partial record;
//   5. a second launch (one workgroup per unit) loads every partial with coalesced vector
//      loads, merges them by log-sum-exp, rotates the rank-space sum back with P_V^T (MFMA)
//      and adds the exact part.
// A tile's first token has the largest rank (storage is rank-descending per chunk), which
// bounds its MFMA steps: ceil(r_max/32) score steps and ceil(r_max/16) value blocks.
#include <mutex>

#include "vr_internal.h"

namespace vr {

constexpr int DC_THREADS = 512;
constexpr int DC_WAVES = 8;
constexpr int DC_SEQ = 16;                 // sequences per launch (descriptors in kernargs)
constexpr int DC_REC = 16 + 16 + 16 * D;   // floats per partial record: m, l, acc[16][128]
constexpr int DC_MAX_CPW = 16;            // chunks one workgroup's tile range may touch
constexpr int DC_MAX_REC = 512;            // partial records per (sequence, head, row tile)

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) uint8_t lds_u8;

__device__ __forceinline__ f32x4 mfma16(u32x2 a, u32x2 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(s16x4, a),
                                                     __builtin_bit_cast(s16x4, b), c, 0, 0, 0);
}

struct DecSeq {
    const void* coef_k;
    const void* coef_v;
    const uint8_t* srank;
    const uint32_t* chunk_off;
    const void* k_exact;
    const void* v_exact;
    const void* q;
    void* out;
    int64_t n_exact;
    const uint32_t* sidx;    // rotary keys: stored position -> token (its position)
};

struct DecParams {
    DecSeq seq[DC_SEQ];
    const float* PK;
    const float* PV;
    float* part;
    int64_t N, coef_stride, cap;
    int G, H, hpg, nqt, rows_total, n_chunks, cpw, n_wg, tpw, total_tiles, units;
    int nrec;                // records per unit (n_wg + 1, plus the anchor records of the residual codec)
    const float* xbar;       // residual codec: [unit][16 total_tiles][ns] anchor-mean score terms
    float* S;                // residual codec: [unit][16 total_tiles][ns] the coded tokens' scores
    int ns;                  // query rows per unit those arrays hold
    const u32x4* rfrag;      // rotary keys: key-basis fragments [G][4][8][2][64] (bf16 hi, lo)
    const float* rfreq;      // rotary keys: theta / (2 pi) per pair as (hi, lo) [128]
    int wpu;                 // ring kernel: workgroups per unit
    int n_xw;                // ring kernel: waves of the unit's last workgroup that take the exact rows
};

template <bool F32> struct Elem;
template <> struct Elem<false> { typedef uint16_t T; };
template <> struct Elem<true> { typedef float T; };

// 4 fp32 -> bf16x4 (hi, lo)
__device__ __forceinline__ void split4(const float* x, u32x2& hi, u32x2& lo) {
    uint32_t h0, l0, h1, l1;
    split2(x[0], x[1], h0, l0);
    split2(x[2], x[3], h1, l1);
    hi = u32x2{h0, h1};
    lo = u32x2{l0, l1};
}

// Staging: each round copies a contiguous coefficient range of both streams (K and V share
// one layout) into LDS with direct-to-LDS 16-byte loads, every unit of the round in flight
// at once; the waves then run their tiles from LDS.
constexpr int DC_STAGE_BYTES = 16384;                         // per stream, round and buffer
constexpr int DC_STAGE_PAD = 64;                              // over-read slack of row gathers
constexpr int DC_LPR = 2 * DC_STAGE_BYTES / 1024 / DC_WAVES;  // loads per wave per round (K and V)
constexpr int DC_TO = 18;                                     // tile offsets per chunk: 17, padded
constexpr int DC_CROW = D + 4;                                // comb row stride (floats)
constexpr int DC_ZERO_BF16 = DC_STAGE_BYTES / 2;               // V stage element in the zeroed pad
typedef unsigned short us2 __attribute__((ext_vector_type(2)));

struct DecSmem {
    uint8_t* stK;     // [2][DC_STAGE_BYTES + pad] staged K coefficients, two rounds in flight;
    uint8_t* stV;     //   [2][..] V; after the tiles: per-wave partial sums comb [4][nr4][128] f32
    float* comb;
    u32x4* qf;        // [4 steps][hi, lo][64 lanes] score B-operand fragments
    float* cm;        // [8][16]
    float* cl;        // [8][16]
    float* mrow;      // [16]
    float* lrow;      // [16]
    int* cT;          // [DC_MAX_CPW] valid tokens per chunk
    uint32_t* cb;     // [DC_MAX_CPW] chunk bases (chunk_off)
    u32x4* kmask;     // [9] bf16 masks keeping the first nv elements of an 8-element row piece
    uint16_t* to;     // [cpw][DC_TO] element offset of tile h inside its chunk, h = 0..16
    uint8_t* mq;      // [cpw][DC_TO] quantised layout: tile h's coordinate count (its rank
                      //   rounded up to a multiple of 8)
    float* rf;        // rotary keys: [128] theta / (2 pi) per pair (hi, lo)
    u32x4* pfr;       // rotary keys: key-basis fragments [4 steps][8 blocks][hi, lo][64 lanes]
    uint8_t* dpos;    // rotary keys: [DC_MAX_CPW][CHUNK] token of each stored position minus
                      //   its chunk's first token
};

__device__ __forceinline__ DecSmem carve(uint8_t* smem) {
    DecSmem s;
    uint8_t* b = smem;
    s.stK = b; b += 2 * (DC_STAGE_BYTES + DC_STAGE_PAD);
    s.stV = b; b += 2 * (DC_STAGE_BYTES + DC_STAGE_PAD);
    s.comb = reinterpret_cast<float*>(s.stK);
    s.qf = reinterpret_cast<u32x4*>(b); b += 4 * 2 * 64 * 16;
    float* f = reinterpret_cast<float*>(b);
    s.cm = f; f += DC_WAVES * 16;
    s.cl = f; f += DC_WAVES * 16;
    s.mrow = f; f += 16;
    s.lrow = f; f += 16;
    s.cT = reinterpret_cast<int*>(f); f += DC_MAX_CPW;
    s.cb = reinterpret_cast<uint32_t*>(f); f += DC_MAX_CPW;
    s.kmask = reinterpret_cast<u32x4*>(f); f += 9 * 4;
    s.rf = f; f += D;
    s.dpos = reinterpret_cast<uint8_t*>(f);
    s.to = reinterpret_cast<uint16_t*>(s.dpos + (size_t)DC_MAX_CPW * CHUNK);
    s.mq = reinterpret_cast<uint8_t*>(s.to + DC_MAX_CPW * DC_TO);
    s.pfr = reinterpret_cast<u32x4*>(s.mq + DC_MAX_CPW * DC_TO);   // 16-byte aligned offset
    return s;
}
constexpr size_t DC_RFRAG_BYTES = (size_t)4 * 8 * 2 * 64 * 16;     // 64 KB

// (the small rotary tables are carved for every variant, so one layout serves all; the
// fragments only in the rotary variant, which then runs one workgroup per CU)
static inline size_t decode_smem_bytes(int cpw, bool rope = false) {
    (void)cpw;
    return 4 * (size_t)(DC_STAGE_BYTES + DC_STAGE_PAD) + 4 * 2 * 64 * 16 +
           (size_t)(2 * DC_WAVES * 16 + 32 + 2 * DC_MAX_CPW + 9 * 4 + D) * 4 + (size_t)DC_MAX_CPW * CHUNK +
           (size_t)DC_MAX_CPW * DC_TO * 2 + (size_t)DC_MAX_CPW * DC_TO + (rope ? DC_RFRAG_BYTES : 0);
}

// 8 consecutive bf16 at element index a of an LDS array (any 2-byte alignment): five dword
// reads realigned by a funnel shift.
__device__ __forceinline__ u32x4 lds_row8_bf16(const uint32_t* w, int a) {
    const int w0 = a >> 1;
    const uint32_t sh = (uint32_t)(a & 1) * 16u;
    const uint32_t d0 = w[w0], d1 = w[w0 + 1], d2 = w[w0 + 2], d3 = w[w0 + 3], d4 = w[w0 + 4];
    return u32x4{__builtin_amdgcn_alignbit(d1, d0, sh), __builtin_amdgcn_alignbit(d2, d1, sh),
                 __builtin_amdgcn_alignbit(d3, d2, sh), __builtin_amdgcn_alignbit(d4, d3, sh)};
}

// Inclusive prefix sum over the 16 lanes of each DPP row (lanes 16 r .. 16 r + 15).
__device__ __forceinline__ uint32_t row_scan16(uint32_t x) {
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x111, 0xf, 0xf, true);   // row_shr:1
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x112, 0xf, 0xf, true);   // row_shr:2
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x114, 0xf, 0xf, true);   // row_shr:4
    x += (uint32_t)__builtin_amdgcn_update_dpp(0, (int)x, 0x118, 0xf, 0xf, true);   // row_shr:8
    return x;
}

// Lane index, recomputed where it is used (two mbcnt ALU ops).  Volatile asm keeps the
// compiler from merging the instances into one value that would stay live (and be spilled)
// across the tile loop.
__device__ __forceinline__ int lane_now() {
    int l;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
    return l;
}

// The value-product accumulators O^T (8 blocks of 16 rank coordinates x 16 query rows, one
// f32x4 per lane per block) live in AGPRs a0..a31 for the whole tile loop: block b in
// a[4b .. 4b + 3].  The MFMAs that update them, their rare rescale and the final read-out
// are inline asm naming those registers, so the compiler never moves them between
// registers at the joins of the tile loop (which it otherwise does with a copy of all 32
// accumulators per tile).  Every statement lists them as clobbered, so the kernel's
// register allocation counts them and the compiler keeps nothing of its own there.
// Hazards are padded by hand: 2 wait states from a VALU write of an operand to the first
// MFMA, 24 from the last MFMA to a VALU read of its result, 5 from an AGPR write by VALU to
// an MFMA that accumulates into it.
#define ACC_AGPRS "a0", "a1", "a2", "a3", "a4", "a5", "a6", "a7", "a8", "a9", "a10", "a11", "a12", "a13", "a14", "a15", "a16", "a17", "a18", "a19", "a20", "a21", "a22", "a23", "a24", "a25", "a26", "a27", "a28", "a29", "a30", "a31"
__device__ __forceinline__ void acc_zero() {
    asm volatile("v_accvgpr_write_b32 a0, 0\n\t" "v_accvgpr_write_b32 a1, 0\n\t" "v_accvgpr_write_b32 a2, 0\n\t" "v_accvgpr_write_b32 a3, 0\n\t" "v_accvgpr_write_b32 a4, 0\n\t" "v_accvgpr_write_b32 a5, 0\n\t" "v_accvgpr_write_b32 a6, 0\n\t" "v_accvgpr_write_b32 a7, 0\n\t" "v_accvgpr_write_b32 a8, 0\n\t" "v_accvgpr_write_b32 a9, 0\n\t" "v_accvgpr_write_b32 a10, 0\n\t" "v_accvgpr_write_b32 a11, 0\n\t" "v_accvgpr_write_b32 a12, 0\n\t" "v_accvgpr_write_b32 a13, 0\n\t" "v_accvgpr_write_b32 a14, 0\n\t" "v_accvgpr_write_b32 a15, 0\n\t" "v_accvgpr_write_b32 a16, 0\n\t" "v_accvgpr_write_b32 a17, 0\n\t" "v_accvgpr_write_b32 a18, 0\n\t" "v_accvgpr_write_b32 a19, 0\n\t" "v_accvgpr_write_b32 a20, 0\n\t" "v_accvgpr_write_b32 a21, 0\n\t" "v_accvgpr_write_b32 a22, 0\n\t" "v_accvgpr_write_b32 a23, 0\n\t" "v_accvgpr_write_b32 a24, 0\n\t" "v_accvgpr_write_b32 a25, 0\n\t" "v_accvgpr_write_b32 a26, 0\n\t" "v_accvgpr_write_b32 a27, 0\n\t" "v_accvgpr_write_b32 a28, 0\n\t" "v_accvgpr_write_b32 a29, 0\n\t" "v_accvgpr_write_b32 a30, 0\n\t" "v_accvgpr_write_b32 a31, 0\n\t" "s_nop 4\n\t" ::: ACC_AGPRS);
}
template <int NB> __device__ __forceinline__ void acc_mfma_bf16(const u32x2* vh, u32x2 ph);
template <> __device__ __forceinline__ void acc_mfma_bf16<1>(const u32x2* vh, u32x2 ph) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %1, a[0:3]\n\t" :: "v"(vh[0]), "v"(ph) : ACC_AGPRS);
}
template <> __device__ __forceinline__ void acc_mfma_bf16<2>(const u32x2* vh, u32x2 ph) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %2, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %1, %2, a[4:7]\n\t" :: "v"(vh[0]), "v"(vh[1]), "v"(ph) : ACC_AGPRS);
}
template <> __device__ __forceinline__ void acc_mfma_bf16<4>(const u32x2* vh, u32x2 ph) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %4, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %1, %4, a[4:7]\n\t" "v_mfma_f32_16x16x16_bf16 a[8:11], %2, %4, a[8:11]\n\t" "v_mfma_f32_16x16x16_bf16 a[12:15], %3, %4, a[12:15]\n\t" :: "v"(vh[0]), "v"(vh[1]), "v"(vh[2]), "v"(vh[3]), "v"(ph) : ACC_AGPRS);
}
template <> __device__ __forceinline__ void acc_mfma_bf16<8>(const u32x2* vh, u32x2 ph) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %8, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %1, %8, a[4:7]\n\t" "v_mfma_f32_16x16x16_bf16 a[8:11], %2, %8, a[8:11]\n\t" "v_mfma_f32_16x16x16_bf16 a[12:15], %3, %8, a[12:15]\n\t" "v_mfma_f32_16x16x16_bf16 a[16:19], %4, %8, a[16:19]\n\t" "v_mfma_f32_16x16x16_bf16 a[20:23], %5, %8, a[20:23]\n\t" "v_mfma_f32_16x16x16_bf16 a[24:27], %6, %8, a[24:27]\n\t" "v_mfma_f32_16x16x16_bf16 a[28:31], %7, %8, a[28:31]\n\t" :: "v"(vh[0]), "v"(vh[1]), "v"(vh[2]), "v"(vh[3]), "v"(vh[4]), "v"(vh[5]), "v"(vh[6]), "v"(vh[7]), "v"(ph) : ACC_AGPRS);
}
template <int NB> __device__ __forceinline__ void acc_mfma_f32(const u32x2* vh, const u32x2* vl, u32x2 ph, u32x2 pl);
template <> __device__ __forceinline__ void acc_mfma_f32<1>(const u32x2* vh, const u32x2* vl, u32x2 ph, u32x2 pl) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %2, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %3, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %1, %2, a[0:3]\n\t" :: "v"(vh[0]), "v"(vl[0]), "v"(ph), "v"(pl) : ACC_AGPRS);
}
template <> __device__ __forceinline__ void acc_mfma_f32<2>(const u32x2* vh, const u32x2* vl, u32x2 ph, u32x2 pl) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %4, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %5, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %2, %4, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %1, %4, a[4:7]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %1, %5, a[4:7]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %3, %4, a[4:7]\n\t" :: "v"(vh[0]), "v"(vh[1]), "v"(vl[0]), "v"(vl[1]), "v"(ph), "v"(pl) : ACC_AGPRS);
}
template <> __device__ __forceinline__ void acc_mfma_f32<4>(const u32x2* vh, const u32x2* vl, u32x2 ph, u32x2 pl) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %8, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %9, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %4, %8, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %1, %8, a[4:7]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %1, %9, a[4:7]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %5, %8, a[4:7]\n\t" "v_mfma_f32_16x16x16_bf16 a[8:11], %2, %8, a[8:11]\n\t" "v_mfma_f32_16x16x16_bf16 a[8:11], %2, %9, a[8:11]\n\t" "v_mfma_f32_16x16x16_bf16 a[8:11], %6, %8, a[8:11]\n\t" "v_mfma_f32_16x16x16_bf16 a[12:15], %3, %8, a[12:15]\n\t" "v_mfma_f32_16x16x16_bf16 a[12:15], %3, %9, a[12:15]\n\t" "v_mfma_f32_16x16x16_bf16 a[12:15], %7, %8, a[12:15]\n\t" :: "v"(vh[0]), "v"(vh[1]), "v"(vh[2]), "v"(vh[3]), "v"(vl[0]), "v"(vl[1]), "v"(vl[2]), "v"(vl[3]), "v"(ph), "v"(pl) : ACC_AGPRS);
}
template <> __device__ __forceinline__ void acc_mfma_f32<8>(const u32x2* vh, const u32x2* vl, u32x2 ph, u32x2 pl) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %16, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %17, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %8, %16, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %1, %16, a[4:7]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %1, %17, a[4:7]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %9, %16, a[4:7]\n\t" "v_mfma_f32_16x16x16_bf16 a[8:11], %2, %16, a[8:11]\n\t" "v_mfma_f32_16x16x16_bf16 a[8:11], %2, %17, a[8:11]\n\t" "v_mfma_f32_16x16x16_bf16 a[8:11], %10, %16, a[8:11]\n\t" "v_mfma_f32_16x16x16_bf16 a[12:15], %3, %16, a[12:15]\n\t" "v_mfma_f32_16x16x16_bf16 a[12:15], %3, %17, a[12:15]\n\t" "v_mfma_f32_16x16x16_bf16 a[12:15], %11, %16, a[12:15]\n\t" "v_mfma_f32_16x16x16_bf16 a[16:19], %4, %16, a[16:19]\n\t" "v_mfma_f32_16x16x16_bf16 a[16:19], %4, %17, a[16:19]\n\t" "v_mfma_f32_16x16x16_bf16 a[16:19], %12, %16, a[16:19]\n\t" "v_mfma_f32_16x16x16_bf16 a[20:23], %5, %16, a[20:23]\n\t" "v_mfma_f32_16x16x16_bf16 a[20:23], %5, %17, a[20:23]\n\t" "v_mfma_f32_16x16x16_bf16 a[20:23], %13, %16, a[20:23]\n\t" "v_mfma_f32_16x16x16_bf16 a[24:27], %6, %16, a[24:27]\n\t" "v_mfma_f32_16x16x16_bf16 a[24:27], %6, %17, a[24:27]\n\t" "v_mfma_f32_16x16x16_bf16 a[24:27], %14, %16, a[24:27]\n\t" "v_mfma_f32_16x16x16_bf16 a[28:31], %7, %16, a[28:31]\n\t" "v_mfma_f32_16x16x16_bf16 a[28:31], %7, %17, a[28:31]\n\t" "v_mfma_f32_16x16x16_bf16 a[28:31], %15, %16, a[28:31]\n\t" :: "v"(vh[0]), "v"(vh[1]), "v"(vh[2]), "v"(vh[3]), "v"(vh[4]), "v"(vh[5]), "v"(vh[6]), "v"(vh[7]), "v"(vl[0]), "v"(vl[1]), "v"(vl[2]), "v"(vl[3]), "v"(vl[4]), "v"(vl[5]), "v"(vl[6]), "v"(vl[7]), "v"(ph), "v"(pl) : ACC_AGPRS);
}
__device__ __forceinline__ void acc_scale(float alpha) {
    float t0, t1, t2, t3;
    asm volatile("s_nop 15\n\ts_nop 7\n\t" "v_accvgpr_read_b32 %0, a0\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a0, %0\n\t" "v_accvgpr_read_b32 %1, a1\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a1, %1\n\t" "v_accvgpr_read_b32 %2, a2\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a2, %2\n\t" "v_accvgpr_read_b32 %3, a3\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a3, %3\n\t" "v_accvgpr_read_b32 %0, a4\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a4, %0\n\t" "v_accvgpr_read_b32 %1, a5\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a5, %1\n\t" "v_accvgpr_read_b32 %2, a6\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a6, %2\n\t" "v_accvgpr_read_b32 %3, a7\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a7, %3\n\t" "v_accvgpr_read_b32 %0, a8\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a8, %0\n\t" "v_accvgpr_read_b32 %1, a9\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a9, %1\n\t" "v_accvgpr_read_b32 %2, a10\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a10, %2\n\t" "v_accvgpr_read_b32 %3, a11\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a11, %3\n\t" "v_accvgpr_read_b32 %0, a12\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a12, %0\n\t" "v_accvgpr_read_b32 %1, a13\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a13, %1\n\t" "v_accvgpr_read_b32 %2, a14\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a14, %2\n\t" "v_accvgpr_read_b32 %3, a15\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a15, %3\n\t" "v_accvgpr_read_b32 %0, a16\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a16, %0\n\t" "v_accvgpr_read_b32 %1, a17\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a17, %1\n\t" "v_accvgpr_read_b32 %2, a18\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a18, %2\n\t" "v_accvgpr_read_b32 %3, a19\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a19, %3\n\t" "v_accvgpr_read_b32 %0, a20\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a20, %0\n\t" "v_accvgpr_read_b32 %1, a21\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a21, %1\n\t" "v_accvgpr_read_b32 %2, a22\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a22, %2\n\t" "v_accvgpr_read_b32 %3, a23\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a23, %3\n\t" "v_accvgpr_read_b32 %0, a24\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a24, %0\n\t" "v_accvgpr_read_b32 %1, a25\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a25, %1\n\t" "v_accvgpr_read_b32 %2, a26\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a26, %2\n\t" "v_accvgpr_read_b32 %3, a27\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a27, %3\n\t" "v_accvgpr_read_b32 %0, a28\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a28, %0\n\t" "v_accvgpr_read_b32 %1, a29\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a29, %1\n\t" "v_accvgpr_read_b32 %2, a30\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a30, %2\n\t" "v_accvgpr_read_b32 %3, a31\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a31, %3\n\t" "s_nop 4\n\t" : "=&v"(t0), "=&v"(t1), "=&v"(t2), "=&v"(t3) : "v"(alpha) : ACC_AGPRS);
}
__device__ __forceinline__ void acc_read(f32x4 (&acc)[8]) {
    asm volatile("s_nop 15\n\ts_nop 7\n\t" "v_accvgpr_read_b32 %0, a0\n\t" "v_accvgpr_read_b32 %1, a1\n\t" "v_accvgpr_read_b32 %2, a2\n\t" "v_accvgpr_read_b32 %3, a3\n\t" "v_accvgpr_read_b32 %4, a4\n\t" "v_accvgpr_read_b32 %5, a5\n\t" "v_accvgpr_read_b32 %6, a6\n\t" "v_accvgpr_read_b32 %7, a7\n\t" "v_accvgpr_read_b32 %8, a8\n\t" "v_accvgpr_read_b32 %9, a9\n\t" "v_accvgpr_read_b32 %10, a10\n\t" "v_accvgpr_read_b32 %11, a11\n\t" "v_accvgpr_read_b32 %12, a12\n\t" "v_accvgpr_read_b32 %13, a13\n\t" "v_accvgpr_read_b32 %14, a14\n\t" "v_accvgpr_read_b32 %15, a15\n\t" "v_accvgpr_read_b32 %16, a16\n\t" "v_accvgpr_read_b32 %17, a17\n\t" "v_accvgpr_read_b32 %18, a18\n\t" "v_accvgpr_read_b32 %19, a19\n\t" "v_accvgpr_read_b32 %20, a20\n\t" "v_accvgpr_read_b32 %21, a21\n\t" "v_accvgpr_read_b32 %22, a22\n\t" "v_accvgpr_read_b32 %23, a23\n\t" "v_accvgpr_read_b32 %24, a24\n\t" "v_accvgpr_read_b32 %25, a25\n\t" "v_accvgpr_read_b32 %26, a26\n\t" "v_accvgpr_read_b32 %27, a27\n\t" "v_accvgpr_read_b32 %28, a28\n\t" "v_accvgpr_read_b32 %29, a29\n\t" "v_accvgpr_read_b32 %30, a30\n\t" "v_accvgpr_read_b32 %31, a31\n\t" : "=v"(acc[0][0]), "=v"(acc[0][1]), "=v"(acc[0][2]), "=v"(acc[0][3]), "=v"(acc[1][0]), "=v"(acc[1][1]), "=v"(acc[1][2]), "=v"(acc[1][3]), "=v"(acc[2][0]), "=v"(acc[2][1]), "=v"(acc[2][2]), "=v"(acc[2][3]), "=v"(acc[3][0]), "=v"(acc[3][1]), "=v"(acc[3][2]), "=v"(acc[3][3]), "=v"(acc[4][0]), "=v"(acc[4][1]), "=v"(acc[4][2]), "=v"(acc[4][3]), "=v"(acc[5][0]), "=v"(acc[5][1]), "=v"(acc[5][2]), "=v"(acc[5][3]), "=v"(acc[6][0]), "=v"(acc[6][1]), "=v"(acc[6][2]), "=v"(acc[6][3]), "=v"(acc[7][0]), "=v"(acc[7][1]), "=v"(acc[7][2]), "=v"(acc[7][3]) :: ACC_AGPRS);
}

// The second set of accumulators (a32..a63), for a wave that serves two row tiles of query
// rows at once: the same helpers on the other registers.
#define ACC1_AGPRS "a32", "a33", "a34", "a35", "a36", "a37", "a38", "a39", "a40", "a41", "a42", "a43", "a44", "a45", "a46", "a47", "a48", "a49", "a50", "a51", "a52", "a53", "a54", "a55", "a56", "a57", "a58", "a59", "a60", "a61", "a62", "a63"
__device__ __forceinline__ void acc1_zero() {
    asm volatile("v_accvgpr_write_b32 a32, 0\n\t" "v_accvgpr_write_b32 a33, 0\n\t" "v_accvgpr_write_b32 a34, 0\n\t" "v_accvgpr_write_b32 a35, 0\n\t" "v_accvgpr_write_b32 a36, 0\n\t" "v_accvgpr_write_b32 a37, 0\n\t" "v_accvgpr_write_b32 a38, 0\n\t" "v_accvgpr_write_b32 a39, 0\n\t" "v_accvgpr_write_b32 a40, 0\n\t" "v_accvgpr_write_b32 a41, 0\n\t" "v_accvgpr_write_b32 a42, 0\n\t" "v_accvgpr_write_b32 a43, 0\n\t" "v_accvgpr_write_b32 a44, 0\n\t" "v_accvgpr_write_b32 a45, 0\n\t" "v_accvgpr_write_b32 a46, 0\n\t" "v_accvgpr_write_b32 a47, 0\n\t" "v_accvgpr_write_b32 a48, 0\n\t" "v_accvgpr_write_b32 a49, 0\n\t" "v_accvgpr_write_b32 a50, 0\n\t" "v_accvgpr_write_b32 a51, 0\n\t" "v_accvgpr_write_b32 a52, 0\n\t" "v_accvgpr_write_b32 a53, 0\n\t" "v_accvgpr_write_b32 a54, 0\n\t" "v_accvgpr_write_b32 a55, 0\n\t" "v_accvgpr_write_b32 a56, 0\n\t" "v_accvgpr_write_b32 a57, 0\n\t" "v_accvgpr_write_b32 a58, 0\n\t" "v_accvgpr_write_b32 a59, 0\n\t" "v_accvgpr_write_b32 a60, 0\n\t" "v_accvgpr_write_b32 a61, 0\n\t" "v_accvgpr_write_b32 a62, 0\n\t" "v_accvgpr_write_b32 a63, 0\n\t" "s_nop 4\n\t" ::: ACC1_AGPRS);
}
template <int NB> __device__ __forceinline__ void acc1_mfma_bf16(const u32x2* vh, u32x2 ph);
template <> __device__ __forceinline__ void acc1_mfma_bf16<1>(const u32x2* vh, u32x2 ph) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[32:35], %0, %1, a[32:35]\n\t" :: "v"(vh[0]), "v"(ph) : ACC1_AGPRS);
}
template <> __device__ __forceinline__ void acc1_mfma_bf16<2>(const u32x2* vh, u32x2 ph) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[32:35], %0, %2, a[32:35]\n\t" "v_mfma_f32_16x16x16_bf16 a[36:39], %1, %2, a[36:39]\n\t" :: "v"(vh[0]), "v"(vh[1]), "v"(ph) : ACC1_AGPRS);
}
template <> __device__ __forceinline__ void acc1_mfma_bf16<4>(const u32x2* vh, u32x2 ph) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[32:35], %0, %4, a[32:35]\n\t" "v_mfma_f32_16x16x16_bf16 a[36:39], %1, %4, a[36:39]\n\t" "v_mfma_f32_16x16x16_bf16 a[40:43], %2, %4, a[40:43]\n\t" "v_mfma_f32_16x16x16_bf16 a[44:47], %3, %4, a[44:47]\n\t" :: "v"(vh[0]), "v"(vh[1]), "v"(vh[2]), "v"(vh[3]), "v"(ph) : ACC1_AGPRS);
}
template <> __device__ __forceinline__ void acc1_mfma_bf16<8>(const u32x2* vh, u32x2 ph) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[32:35], %0, %8, a[32:35]\n\t" "v_mfma_f32_16x16x16_bf16 a[36:39], %1, %8, a[36:39]\n\t" "v_mfma_f32_16x16x16_bf16 a[40:43], %2, %8, a[40:43]\n\t" "v_mfma_f32_16x16x16_bf16 a[44:47], %3, %8, a[44:47]\n\t" "v_mfma_f32_16x16x16_bf16 a[48:51], %4, %8, a[48:51]\n\t" "v_mfma_f32_16x16x16_bf16 a[52:55], %5, %8, a[52:55]\n\t" "v_mfma_f32_16x16x16_bf16 a[56:59], %6, %8, a[56:59]\n\t" "v_mfma_f32_16x16x16_bf16 a[60:63], %7, %8, a[60:63]\n\t" :: "v"(vh[0]), "v"(vh[1]), "v"(vh[2]), "v"(vh[3]), "v"(vh[4]), "v"(vh[5]), "v"(vh[6]), "v"(vh[7]), "v"(ph) : ACC1_AGPRS);
}
__device__ __forceinline__ void acc1_scale(float alpha) {
    float t0, t1, t2, t3;
    asm volatile("s_nop 15\n\ts_nop 7\n\t" "v_accvgpr_read_b32 %0, a32\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a32, %0\n\t" "v_accvgpr_read_b32 %1, a33\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a33, %1\n\t" "v_accvgpr_read_b32 %2, a34\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a34, %2\n\t" "v_accvgpr_read_b32 %3, a35\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a35, %3\n\t" "v_accvgpr_read_b32 %0, a36\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a36, %0\n\t" "v_accvgpr_read_b32 %1, a37\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a37, %1\n\t" "v_accvgpr_read_b32 %2, a38\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a38, %2\n\t" "v_accvgpr_read_b32 %3, a39\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a39, %3\n\t" "v_accvgpr_read_b32 %0, a40\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a40, %0\n\t" "v_accvgpr_read_b32 %1, a41\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a41, %1\n\t" "v_accvgpr_read_b32 %2, a42\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a42, %2\n\t" "v_accvgpr_read_b32 %3, a43\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a43, %3\n\t" "v_accvgpr_read_b32 %0, a44\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a44, %0\n\t" "v_accvgpr_read_b32 %1, a45\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a45, %1\n\t" "v_accvgpr_read_b32 %2, a46\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a46, %2\n\t" "v_accvgpr_read_b32 %3, a47\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a47, %3\n\t" "v_accvgpr_read_b32 %0, a48\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a48, %0\n\t" "v_accvgpr_read_b32 %1, a49\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a49, %1\n\t" "v_accvgpr_read_b32 %2, a50\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a50, %2\n\t" "v_accvgpr_read_b32 %3, a51\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a51, %3\n\t" "v_accvgpr_read_b32 %0, a52\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a52, %0\n\t" "v_accvgpr_read_b32 %1, a53\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a53, %1\n\t" "v_accvgpr_read_b32 %2, a54\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a54, %2\n\t" "v_accvgpr_read_b32 %3, a55\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a55, %3\n\t" "v_accvgpr_read_b32 %0, a56\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a56, %0\n\t" "v_accvgpr_read_b32 %1, a57\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a57, %1\n\t" "v_accvgpr_read_b32 %2, a58\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a58, %2\n\t" "v_accvgpr_read_b32 %3, a59\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a59, %3\n\t" "v_accvgpr_read_b32 %0, a60\n\tv_mul_f32 %0, %0, %4\n\tv_accvgpr_write_b32 a60, %0\n\t" "v_accvgpr_read_b32 %1, a61\n\tv_mul_f32 %1, %1, %4\n\tv_accvgpr_write_b32 a61, %1\n\t" "v_accvgpr_read_b32 %2, a62\n\tv_mul_f32 %2, %2, %4\n\tv_accvgpr_write_b32 a62, %2\n\t" "v_accvgpr_read_b32 %3, a63\n\tv_mul_f32 %3, %3, %4\n\tv_accvgpr_write_b32 a63, %3\n\t" "s_nop 4\n\t" : "=&v"(t0), "=&v"(t1), "=&v"(t2), "=&v"(t3) : "v"(alpha) : ACC1_AGPRS);
}
__device__ __forceinline__ void acc1_read(f32x4 (&acc)[8]) {
    asm volatile("s_nop 15\n\ts_nop 7\n\t" "v_accvgpr_read_b32 %0, a32\n\t" "v_accvgpr_read_b32 %1, a33\n\t" "v_accvgpr_read_b32 %2, a34\n\t" "v_accvgpr_read_b32 %3, a35\n\t" "v_accvgpr_read_b32 %4, a36\n\t" "v_accvgpr_read_b32 %5, a37\n\t" "v_accvgpr_read_b32 %6, a38\n\t" "v_accvgpr_read_b32 %7, a39\n\t" "v_accvgpr_read_b32 %8, a40\n\t" "v_accvgpr_read_b32 %9, a41\n\t" "v_accvgpr_read_b32 %10, a42\n\t" "v_accvgpr_read_b32 %11, a43\n\t" "v_accvgpr_read_b32 %12, a44\n\t" "v_accvgpr_read_b32 %13, a45\n\t" "v_accvgpr_read_b32 %14, a46\n\t" "v_accvgpr_read_b32 %15, a47\n\t" "v_accvgpr_read_b32 %16, a48\n\t" "v_accvgpr_read_b32 %17, a49\n\t" "v_accvgpr_read_b32 %18, a50\n\t" "v_accvgpr_read_b32 %19, a51\n\t" "v_accvgpr_read_b32 %20, a52\n\t" "v_accvgpr_read_b32 %21, a53\n\t" "v_accvgpr_read_b32 %22, a54\n\t" "v_accvgpr_read_b32 %23, a55\n\t" "v_accvgpr_read_b32 %24, a56\n\t" "v_accvgpr_read_b32 %25, a57\n\t" "v_accvgpr_read_b32 %26, a58\n\t" "v_accvgpr_read_b32 %27, a59\n\t" "v_accvgpr_read_b32 %28, a60\n\t" "v_accvgpr_read_b32 %29, a61\n\t" "v_accvgpr_read_b32 %30, a62\n\t" "v_accvgpr_read_b32 %31, a63\n\t" : "=v"(acc[0][0]), "=v"(acc[0][1]), "=v"(acc[0][2]), "=v"(acc[0][3]), "=v"(acc[1][0]), "=v"(acc[1][1]), "=v"(acc[1][2]), "=v"(acc[1][3]), "=v"(acc[2][0]), "=v"(acc[2][1]), "=v"(acc[2][2]), "=v"(acc[2][3]), "=v"(acc[3][0]), "=v"(acc[3][1]), "=v"(acc[3][2]), "=v"(acc[3][3]), "=v"(acc[4][0]), "=v"(acc[4][1]), "=v"(acc[4][2]), "=v"(acc[4][3]), "=v"(acc[5][0]), "=v"(acc[5][1]), "=v"(acc[5][2]), "=v"(acc[5][3]), "=v"(acc[6][0]), "=v"(acc[6][1]), "=v"(acc[6][2]), "=v"(acc[6][3]), "=v"(acc[7][0]), "=v"(acc[7][1]), "=v"(acc[7][2]), "=v"(acc[7][3]) :: ACC1_AGPRS);
}
// Accumulator set SET (0: a0..a31, 1: a32..a63).
template <int SET> __device__ __forceinline__ void accs_zero() { if constexpr (SET == 0) acc_zero(); else acc1_zero(); }
template <int SET, int NB> __device__ __forceinline__ void accs_mfma_bf16(const u32x2* vh, u32x2 ph) {
    if constexpr (SET == 0) acc_mfma_bf16<NB>(vh, ph); else acc1_mfma_bf16<NB>(vh, ph);
}
template <int SET> __device__ __forceinline__ void accs_scale(float alpha) { if constexpr (SET == 0) acc_scale(alpha); else acc1_scale(alpha); }
template <int SET> __device__ __forceinline__ void accs_read(f32x4 (&acc)[8]) { if constexpr (SET == 0) acc_read(acc); else acc1_read(acc); }

// One 16-position tile in the stage (wave-uniform): its first position i0 inside the chunk
// (or the exact rows), the chunk's valid positions T, the stage offset of its first element
// and its size m (coded: the largest rank of the tile; exact rows: 128).
struct TileMeta {
    int i0, T, base, m;
    const float* xb;   // residual codec: the tile's 16 positions' anchor-mean score terms (else NULL)
    float* sw;         // residual codec: where the tile's scores go
    int ns;            // row stride of both
};

// Residual codec: a coded token's score also holds the mean of its anchors' scores (Eq. 2:
// k_hat = anchor mean + P^T (m . c)); the final scores are kept for the anchors' value weights.
__device__ __forceinline__ void anc_scores_in(const TileMeta& tm, int col, int grp, float (&xv)[4]) {
#pragma unroll
    for (int v = 0; v < 4; ++v) xv[v] = 0.f;
    if (tm.xb && col < tm.ns) {
#pragma unroll
        for (int v = 0; v < 4; ++v) xv[v] = tm.xb[(4 * grp + v) * tm.ns + col];
    }
}
__device__ __forceinline__ void anc_scores_out(const TileMeta& tm, int col, int grp, const float (&sv)[4]) {
    if (tm.xb && col < tm.ns) {
#pragma unroll
        for (int v = 0; v < 4; ++v) tm.sw[(4 * grp + v) * tm.ns + col] = sv[v];
    }
}

// One tile.  Scores S[token][row] by 16x16x32 MFMA over KS steps of 32 coefficients (A =
// the tile's key rows, B = the query fragments); the C fragment (lane = query row, tokens
// 4 grp + v) is the B operand of the value product O^T[j][row] += V^T[j][token] P^T[token][row]
// (16x16x16 MFMA over NB blocks of 16 rank coordinates), so each lane owns one query row
// and the online-softmax rescale is lane-local.  KS and NB bound the tile's largest rank,
// so every LDS read is unconditional (masked by value) and they all issue before the first
// wait.
template <bool F32, bool EXACT, int KS, int NB, bool ANC = false>
__device__ __forceinline__ void tile_step(const TileMeta& tm, bool partial, const typename Elem<F32>::T* sK,
                                          const typename Elem<F32>::T* sV, const u32x4* qf,
                                          const u32x4* kmask, int lane, int grp, float& m_run,
                                          float& l_part) {
    const int col = lane & 15;
    float xv[4] = {0.f, 0.f, 0.f, 0.f};
    if constexpr (ANC) anc_scores_in(tm, col, grp, xv);
    // K rows of a coded tile are m coordinates apart (exact rows: 128) with zeros past each
    // position's rank; a row piece past the row's end (into the next row, the pad or the LDS
    // arrays after the stage) is masked.  V blocks are coordinate-major (coded) or row-major
    // exact rows.  Value operand (A of the value product): lane -> coordinate 16 b + col,
    // positions 4 grp .. 4 grp + 3.
    u32x2 vh[NB], vl[NB];
    auto gather_v = [&]() {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const int j = 16 * b + col;
            if constexpr (EXACT) {
                // rows past the exact slots in use hold no data: masked
                if constexpr (F32) {
                    float f4[4];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float t = sV[tm.base + (4 * grp + e) * D + j];
                        f4[e] = tm.i0 + 4 * grp + e < tm.T ? t : 0.f;
                    }
                    split4(f4, vh[b], vl[b]);
                } else {
                    us2 h[2];
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const int a = tm.i0 + 4 * grp + e < tm.T ? tm.base + (4 * grp + e) * D + j : DC_ZERO_BF16;
                        h[e >> 1][e & 1] = sV[a];
                    }
                    vh[b] = u32x2{__builtin_bit_cast(uint32_t, h[0]), __builtin_bit_cast(uint32_t, h[1])};
                    vl[b] = u32x2{0, 0};
                }
            } else {
                // four consecutive positions at coordinate j; past the tile's size: the zeros
                // after the stage
                if constexpr (F32) {
                    const int a = j < tm.m ? tm.base + 16 * j + 4 * grp : DC_STAGE_BYTES / 4;
                    const f32x4 t = *reinterpret_cast<const f32x4*>(sV + a);
                    const float f4[4] = {t[0], t[1], t[2], t[3]};
                    split4(f4, vh[b], vl[b]);
                } else {
                    const int a = j < tm.m ? tm.base + 16 * j + 4 * grp : DC_ZERO_BF16;
                    vh[b] = *reinterpret_cast<const u32x2*>(sV + a);
                    vl[b] = u32x2{0, 0};
                }
            }
        }
    };
    // small tiles: every read issues up front; full-rank tiles: the value reads wait until
    // the scores are done, to keep the register footprint inside two workgroups per CU
    if constexpr (KS < 4) gather_v();
    // scores: A = the tile's key rows (lane -> token i0 + col, coefficients 32 s + 8 grp ..),
    // B = the query fragments; full-rank tiles run in two halves to bound live registers
    f32x4 sc = {0, 0, 0, 0};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        if (KS >= 4 && s == 2) __builtin_amdgcn_sched_barrier(0);
        const int c0 = 32 * s + 8 * grp;
        int nv = tm.m - c0;
        nv = nv < 0 ? 0 : (nv > 8 ? 8 : nv);
        const int a = tm.base + col * (EXACT ? D : tm.m) + c0;
        u32x4 kh, kl;
        if constexpr (!F32) {
            kh = lds_row8_bf16(reinterpret_cast<const uint32_t*>(sK), a) & kmask[nv];
            kl = u32x4{0, 0, 0, 0};
        } else {
            float x8[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) { const float t = sK[a + e]; x8[e] = e < nv ? t : 0.f; }
            split8(x8, kh, kl);
        }
        const u32x4 qh = qf[(s * 2) * 64 + lane], ql = qf[(s * 2 + 1) * 64 + lane];
        sc = mfma(kh, qh, sc);
        sc = mfma(kh, ql, sc);
        if constexpr (F32) sc = mfma(kl, qh, sc);
    }
    if constexpr (KS >= 4) {
        __builtin_amdgcn_sched_barrier(0);
        gather_v();
    }
    float sv[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) sv[v] = sc[v] + xv[v];
    if constexpr (ANC) anc_scores_out(tm, col, grp, sv);
    if (partial) {
#pragma unroll
        for (int v = 0; v < 4; ++v) sv[v] = tm.i0 + 4 * grp + v < tm.T ? sv[v] : -INFINITY;
    }
    float tmax = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
    tmax = xmax32(xmax16(tmax));
    // Lazy reference: exponents are taken against m_run, which moves only when a score
    // exceeds it by more than 8 (so every p stays below e^8); sums and accumulators always
    // share the reference, so the result is the same softmax.
    // The reference moves for every lane at once, so the (rare) rescale is a wave-uniform
    // branch; lanes whose maximum did not jump scale by 1.
    const bool jump = tmax > m_run + 8.f;                // lane-local: this lane's query row
    if (__builtin_amdgcn_ballot_w64(jump) != 0) {
        const float m_new = jump ? tmax : m_run;
        const float alpha = fast_exp(m_run - m_new);
        l_part *= alpha;
        acc_scale(alpha);
        m_run = m_new;
    }
    float pv[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        pv[v] = fast_exp(sv[v] - m_run);      // exp(-inf) = 0 for masked tokens
        l_part += pv[v];
    }
    if constexpr (F32) {
        u32x2 ph, pl;
        split4(pv, ph, pl);
        acc_mfma_f32<NB>(vh, vl, ph, pl);
    } else {
        // bf16 storage: one bf16 rounding of p (relative 2^-9, far inside the output bound)
        const u32x2 ph = {cvt_bf16x2(pv[0], pv[1]), cvt_bf16x2(pv[2], pv[3])};
        acc_mfma_bf16<NB>(vh, ph);
    }
}

// ----------------------------------------------------------------------------------------
// Rotary keys (Sec. 3.1 "Joint per-token vector"; Algorithm 1, last step).  A coded key is
// pre-RoPE, k = P_K^T (m . c), and must be turned to its token's position p before the score,
// so the rank-space score <P_K q, c> does not apply.  One tile:
//   1. reconstruction by MFMA, K^T[dim][token] = sum_j P_K[j][dim] c[token][j]: A = the basis
//      fragments (bf16 hi + lo, held in LDS for the whole workgroup), B = the tile's key rows
//      as staged (the score A operand of the plain decode); C lane -> token col, dims
//      16 b + 4 grp + v for blocks b = 0..7;
//   2. rotation: dims i and i + 64 (pair i) sit in blocks b and b + 4 of the same lane, so it
//      is lane-local; angles from rope_cs at the token's position;
//   3. scores by 16x16x32 MFMA, A = the rotated keys (lane -> token col; step s2 takes the
//      lane's dims of blocks 2 s2 and 2 s2 + 1 as its 8 k-values, split into bf16 hi + lo),
//      B = the query fragments laid out in the same dim order (hi + lo).  The C fragment is
//      that of the plain decode (lane -> query row, tokens 4 grp + v), so the online softmax
//      and the rank-space value product follow unchanged.
template <bool F32, int KS, int NB>
__device__ __forceinline__ void tile_step_rope(const TileMeta& tm, bool partial, const typename Elem<F32>::T* sK,
                                               const typename Elem<F32>::T* sV, const u32x4* qf,
                                               const u32x4* kmask, const u32x4* pfr,
                                               const float* rf, float pos, int lane, int grp, float& m_run,
                                               float& l_part) {
    const int col = lane & 15;
    u32x2 vh[NB], vl[NB];
    auto gather_v = [&]() {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const int j = 16 * b + col;
            if constexpr (F32) {
                const int a = j < tm.m ? tm.base + 16 * j + 4 * grp : DC_STAGE_BYTES / 4;
                const f32x4 t = *reinterpret_cast<const f32x4*>(sV + a);
                const float f4[4] = {t[0], t[1], t[2], t[3]};
                split4(f4, vh[b], vl[b]);
            } else {
                const int a = j < tm.m ? tm.base + 16 * j + 4 * grp : DC_ZERO_BF16;
                vh[b] = *reinterpret_cast<const u32x2*>(sV + a);
                vl[b] = u32x2{0, 0};
            }
        }
    };
    if constexpr (KS < 4) gather_v();
    // 1. reconstruction
    f32x4 kt[8];
#pragma unroll
    for (int b = 0; b < 8; ++b) kt[b] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const int c0 = 32 * s + 8 * grp;
        int nv = tm.m - c0;
        nv = nv < 0 ? 0 : (nv > 8 ? 8 : nv);
        const int a = tm.base + col * tm.m + c0;
        u32x4 kh, kl;
        if constexpr (!F32) {
            kh = lds_row8_bf16(reinterpret_cast<const uint32_t*>(sK), a) & kmask[nv];
            kl = u32x4{0, 0, 0, 0};
        } else {
            float x8[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) { const float t = sK[a + e]; x8[e] = e < nv ? t : 0.f; }
            split8(x8, kh, kl);
        }
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            const u32x4 ph = pfr[((s * 8 + b) * 2) * 64 + lane], pl = pfr[((s * 8 + b) * 2 + 1) * 64 + lane];
            kt[b] = mfma(ph, kh, kt[b]);
            kt[b] = mfma(pl, kh, kt[b]);
            if constexpr (F32) kt[b] = mfma(ph, kl, kt[b]);
        }
    }
    // 2. rotation to the token's position
#pragma unroll
    for (int b = 0; b < 4; ++b) {
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int i = 16 * b + 4 * grp + v;
            float c, sn;
            rope_cs(pos, rf[2 * i], rf[2 * i + 1], c, sn);
            const float x = kt[b][v], y = kt[b + 4][v];
            kt[b][v] = x * c - y * sn;
            kt[b + 4][v] = x * sn + y * c;
        }
    }
    // 3. scores
    f32x4 sc = {0, 0, 0, 0};
#pragma unroll
    for (int s2 = 0; s2 < 4; ++s2) {
        const float x8[8] = {kt[2 * s2][0], kt[2 * s2][1], kt[2 * s2][2], kt[2 * s2][3],
                             kt[2 * s2 + 1][0], kt[2 * s2 + 1][1], kt[2 * s2 + 1][2], kt[2 * s2 + 1][3]};
        u32x4 kh, kl;
        split8(x8, kh, kl);
        const u32x4 qh = qf[(s2 * 2) * 64 + lane], ql = qf[(s2 * 2 + 1) * 64 + lane];
        sc = mfma(kh, qh, sc);
        sc = mfma(kh, ql, sc);
        sc = mfma(kl, qh, sc);
    }
    if constexpr (KS >= 4) gather_v();
    float sv[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) sv[v] = sc[v];
    if (partial) {
#pragma unroll
        for (int v = 0; v < 4; ++v) sv[v] = tm.i0 + 4 * grp + v < tm.T ? sv[v] : -INFINITY;
    }
    float tmax = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
    tmax = xmax32(xmax16(tmax));
    const bool jump = tmax > m_run + 8.f;
    if (__builtin_amdgcn_ballot_w64(jump) != 0) {
        const float m_new = jump ? tmax : m_run;
        const float alpha = fast_exp(m_run - m_new);
        l_part *= alpha;
        acc_scale(alpha);
        m_run = m_new;
    }
    float pv[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        pv[v] = fast_exp(sv[v] - m_run);
        l_part += pv[v];
    }
    if constexpr (F32) {
        u32x2 ph, pl;
        split4(pv, ph, pl);
        acc_mfma_f32<NB>(vh, vl, ph, pl);
    } else {
        const u32x2 ph = {cvt_bf16x2(pv[0], pv[1]), cvt_bf16x2(pv[2], pv[3])};
        acc_mfma_bf16<NB>(vh, ph);
    }
}

// ----------------------------------------------------------------------------------------
// Quantised coefficients (group-wise b-bit codes, Sec. 3.3 "Composability").  A coded tile
// of size m is stored with mq = m rounded up to a multiple of 8 coordinates and KS =
// ceil(m / 32) groups per position: K codes (16 rows of mq codes), then K scales ([KS][16]
// binary16), in the K stream; V codes (mq rows of 16 positions), then V scales, in the V
// stream.  Codes are two's complement b-bit fields packed from bit 0 upward; code k of a
// group with scale sc stands for k * sc.  Tile size in 2-byte units:
template <int QB> __host__ __device__ constexpr uint32_t q_tile_units(uint32_t m) {
    return m == 0 ? 0u : ((m + 7u) & ~7u) * (uint32_t)QB + 16u * ((m + 31u) / 32u);
}
// signed b-bit field e of a word
template <int QB> __device__ __forceinline__ float code_f(uint32_t w, int e) {
    return (float)((int32_t)(w << (32 - QB - QB * e)) >> (32 - QB));
}
__device__ __forceinline__ float half_f(uint32_t w, int hi) {
    return (float)__builtin_bit_cast(_Float16, (uint16_t)(hi ? w >> 16 : w));
}

// Value products whose B operand differs per 32-coordinate group: block b (coordinates
// 16 b ..) uses ph[b / 2] (the softmax weights scaled by the positions' V scales of that group).
template <int NB> __device__ __forceinline__ void acc_mfma_q(const u32x2* vh, const u32x2* ph);
template <> __device__ __forceinline__ void acc_mfma_q<1>(const u32x2* vh, const u32x2* ph) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %1, a[0:3]\n\t" :: "v"(vh[0]), "v"(ph[0]) : ACC_AGPRS);
}
template <> __device__ __forceinline__ void acc_mfma_q<2>(const u32x2* vh, const u32x2* ph) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %2, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %1, %2, a[4:7]\n\t" :: "v"(vh[0]), "v"(vh[1]), "v"(ph[0]) : ACC_AGPRS);
}
template <> __device__ __forceinline__ void acc_mfma_q<4>(const u32x2* vh, const u32x2* ph) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %4, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %1, %4, a[4:7]\n\t" "v_mfma_f32_16x16x16_bf16 a[8:11], %2, %5, a[8:11]\n\t" "v_mfma_f32_16x16x16_bf16 a[12:15], %3, %5, a[12:15]\n\t" :: "v"(vh[0]), "v"(vh[1]), "v"(vh[2]), "v"(vh[3]), "v"(ph[0]), "v"(ph[1]) : ACC_AGPRS);
}
template <> __device__ __forceinline__ void acc_mfma_q<8>(const u32x2* vh, const u32x2* ph) {
    asm volatile("s_nop 4\n\t" "v_mfma_f32_16x16x16_bf16 a[0:3], %0, %8, a[0:3]\n\t" "v_mfma_f32_16x16x16_bf16 a[4:7], %1, %8, a[4:7]\n\t" "v_mfma_f32_16x16x16_bf16 a[8:11], %2, %9, a[8:11]\n\t" "v_mfma_f32_16x16x16_bf16 a[12:15], %3, %9, a[12:15]\n\t" "v_mfma_f32_16x16x16_bf16 a[16:19], %4, %10, a[16:19]\n\t" "v_mfma_f32_16x16x16_bf16 a[20:23], %5, %10, a[20:23]\n\t" "v_mfma_f32_16x16x16_bf16 a[24:27], %6, %11, a[24:27]\n\t" "v_mfma_f32_16x16x16_bf16 a[28:31], %7, %11, a[28:31]\n\t" :: "v"(vh[0]), "v"(vh[1]), "v"(vh[2]), "v"(vh[3]), "v"(vh[4]), "v"(vh[5]), "v"(vh[6]), "v"(vh[7]), "v"(ph[0]), "v"(ph[1]), "v"(ph[2]), "v"(ph[3]) : ACC_AGPRS);
}

// One quantised coded tile (tm.base in 2-byte units of the stage, tm.m = mq).  Scores: the
// MFMA takes the integer codes (exact in bf16) against the query fragments, one K group
// (32 coordinates) per step, and each step's result is scaled by the K scales of the four
// tokens a lane holds.  Values: the codes are the A operand as they are, and the scale of
// each token's V group goes into the B operand (softmax weight x scale, one bf16 rounding).
template <int QB, int KS, int NB, bool ANC>
__device__ __forceinline__ void tile_step_q(const TileMeta& tm, bool partial, const uint16_t* sK,
                                            const uint16_t* sV, const u32x4* qf, int lane, int grp,
                                            float& m_run, float& l_part) {
    const int col = lane & 15;
    const int mq = tm.m;
    float xv[4] = {0.f, 0.f, 0.f, 0.f};
    if constexpr (ANC) anc_scores_in(tm, col, grp, xv);
    const uint32_t* wk = reinterpret_cast<const uint32_t*>(sK + tm.base);   // 16-byte aligned
    const uint32_t* wv = reinterpret_cast<const uint32_t*>(sV + tm.base);
    const int sco = mq * QB;                        // scales after the codes, 2-byte units
    // ---- scores
    f32x4 sc = {0, 0, 0, 0};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        const int c0 = 32 * s + 8 * grp;
        const uint32_t bit = (uint32_t)(QB * (col * mq + (c0 < mq ? c0 : 0)));
        u32x4 kh;
        if constexpr (QB == 8) {
            const uint32_t x0 = wk[bit >> 5], x1 = wk[(bit >> 5) + 1];
            kh = u32x4{cvt_bf16x2(code_f<8>(x0, 0), code_f<8>(x0, 1)), cvt_bf16x2(code_f<8>(x0, 2), code_f<8>(x0, 3)),
                       cvt_bf16x2(code_f<8>(x1, 0), code_f<8>(x1, 1)), cvt_bf16x2(code_f<8>(x1, 2), code_f<8>(x1, 3))};
        } else {
            uint32_t x = wk[bit >> 5];
            if constexpr (QB == 3) x = __builtin_amdgcn_alignbit(wk[(bit >> 5) + 1], x, bit & 31);
            kh = u32x4{cvt_bf16x2(code_f<QB>(x, 0), code_f<QB>(x, 1)), cvt_bf16x2(code_f<QB>(x, 2), code_f<QB>(x, 3)),
                       cvt_bf16x2(code_f<QB>(x, 4), code_f<QB>(x, 5)), cvt_bf16x2(code_f<QB>(x, 6), code_f<QB>(x, 7))};
        }
        const uint32_t keep = c0 < mq ? 0xFFFFFFFFu : 0u;
        kh = kh & keep;
        const u32x4 qh = qf[(s * 2) * 64 + lane], ql = qf[(s * 2 + 1) * 64 + lane];
        f32x4 t = {0, 0, 0, 0};
        t = mfma(kh, qh, t);
        t = mfma(kh, ql, t);
        // K scales of tokens 4 grp .. 4 grp + 3 in group s (groups past the tile's: none)
        u32x2 ks = *reinterpret_cast<const u32x2*>(sK + tm.base + sco + 16 * (32 * s < mq ? s : 0) + 4 * grp);
        ks = 32 * s < mq ? ks : u32x2{0, 0};
        sc[0] += t[0] * half_f(ks[0], 0);
        sc[1] += t[1] * half_f(ks[0], 1);
        sc[2] += t[2] * half_f(ks[1], 0);
        sc[3] += t[3] * half_f(ks[1], 1);
    }
    float sv[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) sv[v] = sc[v] + xv[v];
    if constexpr (ANC) anc_scores_out(tm, col, grp, sv);
    if (partial) {
#pragma unroll
        for (int v = 0; v < 4; ++v) sv[v] = tm.i0 + 4 * grp + v < tm.T ? sv[v] : -INFINITY;
    }
    float tmax = fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3]));
    tmax = xmax32(xmax16(tmax));
    const bool jump = tmax > m_run + 8.f;
    if (__builtin_amdgcn_ballot_w64(jump) != 0) {
        const float m_new = jump ? tmax : m_run;
        const float alpha = fast_exp(m_run - m_new);
        l_part *= alpha;
        acc_scale(alpha);
        m_run = m_new;
    }
    float pv[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) {
        pv[v] = fast_exp(sv[v] - m_run);
        l_part += pv[v];
    }
    // the value codes are read only now, so they are not live across the score steps
    __builtin_amdgcn_sched_barrier(0);
    // ---- value operands: coordinate j = 16 b + col, positions 4 grp .. 4 grp + 3
    u32x2 vh[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
        const int j = 16 * b + col;
        // coordinates past the tile read its first row (in bounds) and are masked
        const uint32_t bit = (uint32_t)(QB * (16 * (j < mq ? j : 0) + 4 * grp));
        const uint32_t d0 = wv[bit >> 5];
        uint32_t x;
        if constexpr (QB == 3) x = __builtin_amdgcn_alignbit(wv[(bit >> 5) + 1], d0, bit & 31);
        else x = d0 >> (bit & 31);
        x = j < mq ? x : 0u;
        vh[b] = u32x2{cvt_bf16x2(code_f<QB>(x, 0), code_f<QB>(x, 1)), cvt_bf16x2(code_f<QB>(x, 2), code_f<QB>(x, 3))};
    }
    // B operands: weights x the V scales of the same tokens, per group of 32 coordinates
    constexpr int NG = (NB + 1) / 2;
    u32x2 ph[NG];
#pragma unroll
    for (int s = 0; s < NG; ++s) {
        u32x2 vs = *reinterpret_cast<const u32x2*>(sV + tm.base + sco + 16 * (32 * s < mq ? s : 0) + 4 * grp);
        vs = 32 * s < mq ? vs : u32x2{0, 0};
        ph[s] = u32x2{cvt_bf16x2(pv[0] * half_f(vs[0], 0), pv[1] * half_f(vs[0], 1)),
                      cvt_bf16x2(pv[2] * half_f(vs[1], 0), pv[3] * half_f(vs[1], 1))};
    }
    acc_mfma_q<NB>(vh, ph);
}

// QB = 0: coefficients stored in the layer's dtype; QB = 3, 4, 8: b-bit codes with binary16
// group scales (bf16 layers only).
template <bool F32, int QB, bool ANC, bool ROPE = false>
__global__ __launch_bounds__(DC_THREADS, (F32 || QB || ROPE) ? 2 : 4) void decode_kernel(DecParams p) {
    static_assert(QB == 0 || !F32, "quantised coefficients come from bf16 layers");
    static_assert(!ROPE || (QB == 0 && !ANC), "rotary keys: plain coefficients, no anchors");
    typedef typename Elem<F32>::T ET;
    constexpr int EPU = 16 / (int)sizeof(ET);               // elements per 16-byte unit
    constexpr int SE = DC_STAGE_BYTES / (int)sizeof(ET);     // staged elements per stream
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    // Workgroup -> (unit, x): consecutive workgroups take consecutive units, so the
    // workgroups of one unit (one KV head) land on the same XCD of the round-robin
    // dispatch and share its L2 copy of the key basis.  x = 0 (dispatched first) is the
    // exact-slot workgroup; x >= 1 take the coded tile ranges.
    const int U = p.units;
    const int L = blockIdx.x;
    const int unit = L % U, x = L / U;
    const int sq = unit / (p.G * p.nqt), gq = unit % (p.G * p.nqt);
    const int g = gq / p.nqt, qt = gq % p.nqt;
    const DecSeq& S = p.seq[sq];
    const int rows = min(16, p.rows_total - 16 * qt);
    const int nr4 = (rows + 3) & ~3;
    const bool exact = x == 0;
    // the later-dispatched half of the grid shares CUs with the earlier half: its waves take
    // the higher issue priority through the prologue, so its metadata and first rounds are not
    // queued behind the earlier half's
    if (L >= (int)(gridDim.x >> 1)) __builtin_amdgcn_s_setprio(1);
    const int xc = x - 1;
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));   // scalar
    int lane = lane_now(), tid = 64 * wave + lane, grp = lane >> 4, col = lane & 15;
    DecSmem sm = carve(smem);
    const float scale = 0.08838834764831845f;  // 1/sqrt(128)
    const ET* qsrc = reinterpret_cast<const ET*>(S.q);

    // ---- 1a. issue the basis rows and query rows (raw loads only: nothing here waits, so
    //          the rank loads below issue right behind them; a missing query row reads
    //          row 0 of the head and is masked later)
    const float* P = p.PK + (int64_t)g * D * D;
    const int qrow_l = 16 * qt + col;
    const bool q_ok = qrow_l < p.rows_total;
    const int query_l = q_ok ? qrow_l / p.hpg : 0, hh_l = q_ok ? qrow_l % p.hpg : 0;
    const ET* qv = qsrc + ((int64_t)query_l * p.H + g * p.hpg + hh_l) * D;
    u32x4 pa[4][2];
    u32x4 qr[4][2];
    const int qs_ = tid >> 7, qpart = (tid >> 6) & 1;   // exact: 4 steps x {hi, lo} x 64 lanes
    if (ROPE && !exact) {
        // the query dims of score step qs_ in the rotary order (dims 32 qs_ + 4 grp .. + 3
        // and 32 qs_ + 16 + 4 grp .. + 3); the basis fragments go to LDS below
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
            const ET* src = qv + 32 * qs_ + 16 * hf + 4 * grp;
            if constexpr (F32) qr[0][hf] = load16(src);
            else { const u32x2 t = *reinterpret_cast<const u32x2*>(src); qr[0][hf] = u32x4{t[0], t[1], 0u, 0u}; }
        }
    } else if (!exact) {
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            const float* src = P + (16 * wave + col) * D + 32 * s + 8 * grp;
            pa[s][0] = load16(src);
            pa[s][1] = load16(src + 4);
            const ET* qsrc8 = qv + 32 * s + 8 * grp;
            if constexpr (F32) { qr[s][0] = load16(qsrc8); qr[s][1] = load16(qsrc8 + 4); }
            else qr[s][0] = load16_a2(qsrc8);
        }
    } else {
        const ET* src = qv + 32 * qs_ + 8 * grp;
        if constexpr (F32) { qr[0][0] = load16(src); qr[0][1] = load16(src + 4); }
        else qr[0][0] = load16_a2(src);
    }
    // ---- 1b. stored ranks (16 per thread: thread 16 c + k holds tile k of chunk c) and
    //          chunk bases of the chunks this tile range touches (at most DC_MAX_CPW)
    const int tau0 = exact ? 0 : xc * p.tpw;
    const int tau1 = exact ? 0 : min(tau0 + p.tpw, p.total_tiles);
    const int c_lo = tau0 >> 4;
    const int ncl = exact ? 0 : ((tau1 - 1) >> 4) - c_lo + 1;
    u32x4 rv = {0, 0, 0, 0};
    uint32_t cbv = 0;
    const int64_t t_r = (int64_t)c_lo * CHUNK + (int64_t)tid * 16;
    const bool r_ok = !exact && tid < ncl * (CHUNK / 16);
    if (r_ok && t_r < p.N) rv = load16(S.srank + t_r);     // srank is padded to a multiple of 64
    if (!exact && tid < ncl) cbv = S.chunk_off[c_lo + tid];
    if constexpr (QB != 0) cbv >>= 1;       // quantised chunk bases are in bytes
    // rotary keys: the basis fragments (8 per thread), the frequency table and each stored
    // position's token offset in its chunk
    u32x4 frv[8];
    if (ROPE && !exact) {
        const u32x4* fr = p.rfrag + (int64_t)g * (4 * 8 * 2 * 64);
#pragma unroll
        for (int k = 0; k < 8; ++k) frv[k] = fr[k * DC_THREADS + tid];
    }
    float rfv = 0.f;
    uint32_t dp[8] = {0u, 0u, 0u, 0u, 0u, 0u, 0u, 0u};
    const bool dp_ok = ROPE && !exact && tid < ncl * (CHUNK / 8);
    if (ROPE && !exact) {
        if (tid < D) rfv = p.rfreq[tid];
        if (dp_ok) {
            const int64_t gi0 = (int64_t)c_lo * CHUNK + 8 * tid;
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int64_t gi = gi0 + k;
                dp[k] = gi < p.N ? S.sidx[gi] - (uint32_t)((gi / CHUNK) * CHUNK) : 0u;
            }
        }
    }

    lane = lane_now(); tid = 64 * wave + lane; grp = lane >> 4; col = lane & 15;
    // ---- 1c. offsets of the stored slots inside each chunk: local prefix sums of a
    //          thread's 16 ranks, then a 16-lane scan of the threads of one chunk (one DPP
    //          row); ranks past the chunk's end count as 0
    if (r_ok) {
        // tile k's size m_k = its first rank; offsets inside the chunk by a 16-lane scan
        const int cc = tid >> 4, k = tid & 15;
        const int64_t t0 = (int64_t)(c_lo + cc) * CHUNK;
        const int T = (int)((p.N - t0) < CHUNK ? (p.N - t0) : CHUNK);
        const uint32_t mk = 16 * k < T ? (rv[0] & 0xFFu) : 0u;
        const uint32_t units = QB ? q_tile_units<QB>(mk) : 16u * mk;
        const uint32_t incl = row_scan16(units);
        sm.to[cc * DC_TO + k] = (uint16_t)(incl - units);
        if constexpr (QB != 0) sm.mq[cc * DC_TO + k] = (uint8_t)((mk + 7u) & ~7u);
        if (k == 15) { sm.to[cc * DC_TO + 16] = (uint16_t)incl; sm.cT[cc] = T; }
    }
    if (!exact && tid < ncl) sm.cb[tid] = cbv;
    if (ROPE && !exact) {
#pragma unroll
        for (int k = 0; k < 8; ++k) sm.pfr[k * DC_THREADS + tid] = frv[k];
        if (tid < D) sm.rf[tid] = rfv;
        if (dp_ok) {
            const uint32_t lo4 = dp[0] | (dp[1] << 8) | (dp[2] << 16) | (dp[3] << 24);
            const uint32_t hi4 = dp[4] | (dp[5] << 8) | (dp[6] << 16) | (dp[7] << 24);
            *reinterpret_cast<u32x2*>(sm.dpos + 8 * tid) = u32x2{lo4, hi4};
        }
    }
    // the V stage's pad holds zeros (coordinates past a token's rank read them), and the
    // K-row masks: entry nv keeps the first nv bf16 elements of an 8-element piece
    if (tid < DC_STAGE_PAD / 2)     // the zeroed pad after each V buffer
        reinterpret_cast<uint32_t*>(sm.stV + (tid >> 4) * (DC_STAGE_BYTES + DC_STAGE_PAD) + DC_STAGE_BYTES)[tid & 15] = 0u;
    if (tid >= 64 && tid < 64 + 9) {
        const int nv = tid - 64;
        u32x4 mk;
#pragma unroll
        for (int k = 0; k < 4; ++k) mk[k] = nv >= 2 * k + 2 ? 0xFFFFFFFFu : (nv == 2 * k + 1 ? 0x0000FFFFu : 0u);
        sm.kmask[nv] = mk;
    }
    __syncthreads();

    const int t_first = exact ? 0 : tau0;
    const int t_end = exact ? (int)((S.n_exact + 15) / 16) : tau1;
    const int nexact = (int)S.n_exact;
    const int64_t hoff = exact ? (int64_t)g * p.cap * D : (int64_t)g * p.coef_stride;
    const int limit = exact ? (int)(p.cap * D) : (int)p.coef_stride;   // elements in the head's stream
    const uint8_t* kg = reinterpret_cast<const uint8_t*>(exact ? S.k_exact : S.coef_k) + hoff * (int64_t)sizeof(ET);
    const uint8_t* vg = reinterpret_cast<const uint8_t*>(exact ? S.v_exact : S.coef_v) + hoff * (int64_t)sizeof(ET);
    // element offsets (in the head stream, or the head's exact rows) of tile tau's first
    // token and of the end of its last token
    auto toff = [&](int tau) -> int {
        if (exact) return tau * 16 * D;
        const int cc = (tau >> 4) - c_lo;
        return (int)sm.cb[cc] + sm.to[cc * DC_TO + (tau & 15)];
    };
    auto tend = [&](int tau) -> int {
        if (exact) return min(16 * tau + 16, nexact) * D;
        const int cc = (tau >> 4) - c_lo;
        return (int)sm.cb[cc] + sm.to[cc * DC_TO + (tau & 15) + 1];
    };

    float m_run = -INFINITY, l_part = 0.f;
    acc_zero();

    // ---- 2a. round plans (wave-uniform): tiles [ta, tb) whose span fits one buffer.  The
    //          span is clamped to the head's buffer, so no metadata can send a load past it.
    struct Round { int ta, tb, s0, nu; };
    auto plan = [&](int ta) -> Round {
        Round r{ta, ta, 0, 0};
        if (ta < t_end) {
            r.s0 = __builtin_amdgcn_readfirstlane(toff(ta) & ~(EPU - 1));
            const int ln = lane_now();
            for (;;) {
                const int cand = r.tb + ln;
                const bool fit = cand < t_end && tend(cand) - r.s0 <= SE;
                const uint64_t m = __ballot(fit);
                const int cnt = m == ~0ull ? 64 : __builtin_ctzll(~m);
                r.tb += cnt;
                if (cnt < 64) break;
            }
            int n_ = (tend(r.tb - 1) - r.s0 + EPU - 1) / EPU;
            const int room = r.s0 >= 0 && r.s0 < limit ? (limit - r.s0) / EPU : 0;
            n_ = n_ < 0 ? 0 : (n_ > room ? room : n_);
            n_ = n_ > SE / EPU ? SE / EPU : n_;
            r.nu = __builtin_amdgcn_readfirstlane(n_);
        }
        return r;
    };
    // ---- 2b. a round's units go straight to LDS buffer `buf`: one load moves 64 lanes x 16
    //          bytes to a contiguous 1 KB block; wave w moves blocks w and w + 8 of K and of
    //          V.  Every wave issues exactly DC_LPR loads per round, whatever the round holds
    //          (lanes and blocks past its units reload its last unit into the unused tail of
    //          the buffer), so a wait for "all but the next round's DC_LPR loads" is exact.
    //          Issued in asm, so the compiler adds no wait of its own for them; non-temporal, so
    //          the streamed coefficients leave L2 before the bases and metadata do.
    auto issue = [&](const Round& r, int buf) {
        const uint8_t* kr = kg + (size_t)r.s0 * sizeof(ET);     // wave-uniform round bases
        const uint8_t* vr = vg + (size_t)r.s0 * sizeof(ET);
        const int wv = __builtin_amdgcn_readfirstlane(wave);
        uint8_t* bk = sm.stK + buf * (DC_STAGE_BYTES + DC_STAGE_PAD);
        uint8_t* bv = sm.stV + buf * (DC_STAGE_BYTES + DC_STAGE_PAD);
#pragma unroll
        for (int k = 0; k < DC_STAGE_BYTES / 1024 / DC_WAVES; ++k) {
            const int m = wv + DC_WAVES * k;
            const uint32_t u = (uint32_t)(64 * m + lane_now());
            // past the round's end: the round's last unit, a line this load already fetches
            const uint32_t uu = (int)u < r.nu ? u : (r.nu > 0 ? (uint32_t)(r.nu - 1) : 0u);
            const uint8_t* srck = kr + 16u * uu;
            const uint8_t* srcv = vr + 16u * uu;
            const uint32_t dk = __builtin_amdgcn_readfirstlane((uint32_t)(size_t)(lds_u8*)(bk + 1024 * m));
            const uint32_t dv = __builtin_amdgcn_readfirstlane((uint32_t)(size_t)(lds_u8*)(bv + 1024 * m));
            asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
                         :: "v"(srck), "s"(dk) : "memory", "m0");
            asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
                         :: "v"(srcv), "s"(dv) : "memory", "m0");
        }
    };
    Round cur = plan(t_first);
    issue(cur, 0);
    Round nxt = plan(cur.tb);
    issue(nxt, 1);
    // ---- 2c. while the round is in flight: score-operand fragments of the query rows
    //          (lane -> query row col, K group grp; bf16 hi and lo parts).  The basis and
    //          query loads landed with the rank loads (issued before them), so nothing here
    //          waits for the direct-to-LDS loads.
    uint32_t* qf32 = reinterpret_cast<uint32_t*>(sm.qf);
    if (ROPE && !exact) {
        // rotary keys: fragments of q itself (scaled), k-values in the rotary dim order
        float v8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            const u32x4& w = qr[0][e >> 2];
            float val;
            if constexpr (F32) val = __uint_as_float(w[e & 3]);
            else val = (e & 1) ? bf_hi(w[(e & 3) >> 1]) : bf_lo(w[(e & 3) >> 1]);
            v8[e] = q_ok ? val * scale : 0.f;
        }
        u32x4 hh, ll;
        split8(v8, hh, ll);
        sm.qf[(qs_ * 2 + qpart) * 64 + lane] = qpart ? ll : hh;
    } else if (!exact) {
        // q' = P_K q / sqrt(d) by MFMA; C lane -> query row col, directions 16 wave + 4 grp + v
        u32x4 qb[4][2];
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            if constexpr (F32) {
                float x8[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) x8[e] = q_ok ? __uint_as_float(qr[s][e >> 2][e & 3]) : 0.f;
                split8(x8, qb[s][0], qb[s][1]);
            } else {
                qb[s][0] = q_ok ? qr[s][0] : u32x4{0, 0, 0, 0};
                qb[s][1] = u32x4{0, 0, 0, 0};
            }
        }
        f32x4 c = {0, 0, 0, 0};
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            float a8[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) { a8[e] = __uint_as_float(pa[s][0][e]); a8[4 + e] = __uint_as_float(pa[s][1][e]); }
            u32x4 ah, al;
            split8(a8, ah, al);
            c = mfma(ah, qb[s][0], c);
            c = mfma(al, qb[s][0], c);
            if constexpr (F32) c = mfma(ah, qb[s][1], c);
        }
        // direction j = 16 wave + 4 grp + v is element (j & 7) of K group ((j & 31) >> 3) of
        // step j >> 5: two bf16 pairs per lane, for the hi and the lo fragment
        uint32_t h[4], l[4];
#pragma unroll
        for (int v = 0; v < 4; ++v) split_bf16(c[v] * scale, h[v], l[v]);
        const int s = wave >> 1, gp = 2 * (wave & 1) + (grp >> 1), dw = 2 * (grp & 1);
        *reinterpret_cast<u32x2*>(qf32 + ((s * 2 + 0) * 64 + gp * 16 + col) * 4 + dw) = u32x2{pack2(h[0], h[1]), pack2(h[2], h[3])};
        *reinterpret_cast<u32x2*>(qf32 + ((s * 2 + 1) * 64 + gp * 16 + col) * 4 + dw) = u32x2{pack2(l[0], l[1]), pack2(l[2], l[3])};
    } else {
        float v8[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            float val;
            if constexpr (F32) val = __uint_as_float(qr[0][e >> 2][e & 3]);
            else val = (e & 1) ? bf_hi(qr[0][0][e >> 1]) : bf_lo(qr[0][0][e >> 1]);
            v8[e] = q_ok ? val * scale : 0.f;
        }
        u32x4 hh, ll;
        split8(v8, hh, ll);
        sm.qf[(qs_ * 2 + qpart) * 64 + lane] = qpart ? ll : hh;
    }


    // the raised priority of the later half only speeds its prologue up (its first loads go
    // out with the earlier half's); in the round loop both halves issue at the same priority
    __builtin_amdgcn_s_setprio(0);
    for (int rd = 0;; ++rd) {
        // this wave's loads of round rd have landed (only the next round's are younger),
        // then every wave's
        asm volatile("s_waitcnt vmcnt(%0)" :: "n"(DC_LPR) : "memory");
        __syncthreads();

        // ---- 3. tiles of the round, from LDS buffer rd & 1
        const int buf = rd & 1;
        const ET* sK = reinterpret_cast<const ET*>(sm.stK + buf * (DC_STAGE_BYTES + DC_STAGE_PAD));
        const ET* sV = reinterpret_cast<const ET*>(sm.stV + buf * (DC_STAGE_BYTES + DC_STAGE_PAD));
        const int ta = cur.ta, tbnd = cur.tb, s0 = cur.s0;
        for (int tile = ta + __builtin_amdgcn_readfirstlane(wave); tile < tbnd; tile += DC_WAVES) {
            // lane-derived addresses are recomputed per tile (a few ALU ops) rather than
            // hoisted out of the loop for all four tile shapes and spilled
            const int ln = lane_now();
            const int col = ln & 15, grp = ln >> 4;
            TileMeta tm;
            tm.base = __builtin_amdgcn_readfirstlane(toff(tile) - s0);
            tm.xb = nullptr;
            tm.sw = nullptr;
            tm.ns = p.ns;
            if (ANC && !exact) {
                const int64_t o = ((int64_t)unit * p.total_tiles + tile) * 16 * p.ns;
                tm.xb = p.xbar + o;
                tm.sw = p.S + o;
            }
            if (exact) {
                tm.i0 = tile * 16;
                tm.T = nexact;
                tm.m = D;
                const bool partial = tm.i0 + 16 > tm.T;
                tile_step<F32, true, 4, 8>(tm, partial, sK, sV, sm.qf, sm.kmask, ln, grp, m_run, l_part);
            } else {
                const int cc = (tile >> 4) - c_lo;
                tm.i0 = (tile & 15) * 16;
                tm.T = __builtin_amdgcn_readfirstlane(sm.cT[cc]);
                const uint16_t* to = sm.to + cc * DC_TO + (tile & 15);
                if constexpr (QB != 0) tm.m = __builtin_amdgcn_readfirstlane((int)sm.mq[cc * DC_TO + (tile & 15)]);
                else tm.m = __builtin_amdgcn_readfirstlane(((int)to[1] - (int)to[0]) >> 4);
                // a tile's size bounds its 32-coefficient score steps and 16-wide value
                // blocks, as compile-time bounds (no branches inside)
                const bool partial = __builtin_amdgcn_readfirstlane(tm.i0 + 16 > tm.T ? 1 : 0) != 0;
                if constexpr (ROPE) {
                    const int ip = (tile & 15) * 16 + col;
                    const float pos = (float)(((tile >> 4) * CHUNK) + (int)sm.dpos[cc * CHUNK + ip]);
                    if (tm.m <= 16) tile_step_rope<F32, 1, 1>(tm, partial, sK, sV, sm.qf, sm.kmask, sm.pfr, sm.rf, pos, ln, grp, m_run, l_part);
                    else if (tm.m <= 32) tile_step_rope<F32, 1, 2>(tm, partial, sK, sV, sm.qf, sm.kmask, sm.pfr, sm.rf, pos, ln, grp, m_run, l_part);
                    else if (tm.m <= 64) tile_step_rope<F32, 2, 4>(tm, partial, sK, sV, sm.qf, sm.kmask, sm.pfr, sm.rf, pos, ln, grp, m_run, l_part);
                    else tile_step_rope<F32, 4, 8>(tm, partial, sK, sV, sm.qf, sm.kmask, sm.pfr, sm.rf, pos, ln, grp, m_run, l_part);
                } else if constexpr (QB != 0) {
                    const uint16_t* qK = reinterpret_cast<const uint16_t*>(sK);
                    const uint16_t* qV = reinterpret_cast<const uint16_t*>(sV);
                    if (tm.m <= 16) tile_step_q<QB, 1, 1, ANC>(tm, partial, qK, qV, sm.qf, ln, grp, m_run, l_part);
                    else if (tm.m <= 32) tile_step_q<QB, 1, 2, ANC>(tm, partial, qK, qV, sm.qf, ln, grp, m_run, l_part);
                    else if (tm.m <= 64) tile_step_q<QB, 2, 4, ANC>(tm, partial, qK, qV, sm.qf, ln, grp, m_run, l_part);
                    else tile_step_q<QB, 4, 8, ANC>(tm, partial, qK, qV, sm.qf, ln, grp, m_run, l_part);
                } else {
                    if (tm.m <= 16) tile_step<F32, false, 1, 1, ANC>(tm, partial, sK, sV, sm.qf, sm.kmask, ln, grp, m_run, l_part);
                    else if (tm.m <= 32) tile_step<F32, false, 1, 2, ANC>(tm, partial, sK, sV, sm.qf, sm.kmask, ln, grp, m_run, l_part);
                    else if (tm.m <= 64) tile_step<F32, false, 2, 4, ANC>(tm, partial, sK, sV, sm.qf, sm.kmask, ln, grp, m_run, l_part);
                    else tile_step<F32, false, 4, 8, ANC>(tm, partial, sK, sV, sm.qf, sm.kmask, ln, grp, m_run, l_part);
                }
            }
        }
        if (tbnd >= t_end) break;
        __syncthreads();   // every wave is done with buffer rd & 1
        cur = nxt;
        nxt = plan(cur.tb);
        issue(nxt, buf);
    }
    f32x4 acc[8];
    acc_read(acc);
    // the loads past the last round (into the idle buffer) land before the buffers are reused
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();

    // ---- 4. combine the waves of this workgroup (fixed order).  Lane (col, grp) holds query
    //          row col: running max m_run, its share of the sum, O[col][16 b + 4 grp + v].
    //          comb rows are padded to DC_CROW floats, so the 16 rows' stores hit distinct banks.
    lane = lane_now(); tid = 64 * wave + lane; grp = lane >> 4; col = lane & 15;
    const float lsum = xsum32(xsum16(l_part));
    if (lane < 16) { sm.cm[wave * 16 + col] = m_run; sm.cl[wave * 16 + col] = lsum; }
    __syncthreads();   // also: every wave is done reading the stage, which comb reuses
    if (tid < 16) {
        float M = -INFINITY;
        for (int w = 0; w < DC_WAVES; ++w) M = fmaxf(M, sm.cm[w * 16 + tid]);
        float Ls = 0.f;
        for (int w = 0; w < DC_WAVES; ++w) {
            const float mw = sm.cm[w * 16 + tid];
            Ls += mw == -INFINITY ? 0.f : sm.cl[w * 16 + tid] * fast_exp(mw - M);
        }
        sm.mrow[tid] = M;
        sm.lrow[tid] = Ls;
    }
    __syncthreads();
    const float mrow = sm.mrow[col];
    const float fac = m_run == -INFINITY ? 0.f : fast_exp(m_run - mrow);
    if (wave >= 4 && col < nr4) {
#pragma unroll
        for (int b = 0; b < 8; ++b)
            *reinterpret_cast<f32x4*>(&sm.comb[((wave - 4) * nr4 + col) * DC_CROW + 16 * b + 4 * grp]) = acc[b] * fac;
    }
    __syncthreads();
    if (wave < 4 && col < nr4) {
#pragma unroll
        for (int b = 0; b < 8; ++b) {
            f32x4* dst = reinterpret_cast<f32x4*>(&sm.comb[(wave * nr4 + col) * DC_CROW + 16 * b + 4 * grp]);
            *dst = acc[b] * fac + *dst;
        }
    }
    __syncthreads();
    float* recs = p.part + (int64_t)unit * p.nrec * DC_REC;
    {
        float* rec = recs + (int64_t)x * DC_REC;
        const int n4 = nr4 * D / 4;
        for (int idx = tid; idx < n4; idx += DC_THREADS) {
            const int ci = (idx >> 5) * DC_CROW + 4 * (idx & 31);   // row idx/32, float4 idx%32
            const f32x4 a = *reinterpret_cast<const f32x4*>(sm.comb + ci);
            const f32x4 b = *reinterpret_cast<const f32x4*>(sm.comb + nr4 * DC_CROW + ci);
            const f32x4 c = *reinterpret_cast<const f32x4*>(sm.comb + 2 * nr4 * DC_CROW + ci);
            const f32x4 d = *reinterpret_cast<const f32x4*>(sm.comb + 3 * nr4 * DC_CROW + ci);
            reinterpret_cast<f32x4*>(rec + 32)[idx] = ((a + b) + c) + d;
        }
        if (tid < 16) { rec[tid] = sm.mrow[tid]; rec[16 + tid] = sm.lrow[tid]; }
    }
}


// ----------------------------------------------------------------------------------------
// Ring-streaming decode (bf16 coefficients, the plain codec).  One workgroup of 8 waves per
// CU; the workgroups of a unit (sequence, KV head, row tile) share its stored tiles.  Every
// wave owns a contiguous run of tiles, i.e. one contiguous byte range of the K stream and the
// same range of the V stream, and streams it through a private ring in LDS (8 KB per
// stream): 1 KB direct-to-LDS loads in stream order, as far ahead of the tile being scored as
// the ring allows.  A wave waits only on its own load counter, so nothing in the tile loop
// waits for another wave.  A tile that crosses the ring's end is gathered with wrapped
// addresses.  The last n_xw waves of the unit's last workgroup attend to the exact rows in
// the original space.  Each workgroup writes its records in the layout the merge launch
// reads: record 0 the exact rows (last workgroup), record 1 + j the coded tiles of
// workgroup j.
constexpr int DR_WAVES = 8;
constexpr int DR_THREADS = 64 * DR_WAVES;
constexpr int DR_RING = 8192;                     // bytes per stream and wave
constexpr int DR_RING_E = DR_RING / 2;            // bf16 elements
constexpr int DR_UNIT = 1024;                     // one load: 64 lanes x 16 bytes
constexpr int DR_NU = DR_RING / DR_UNIT;          // ring slots
constexpr int DR_PAD = 64;                        // zeros after each ring (V reads past a tile's size)
constexpr int DR_RS = DR_RING + DR_PAD;           // ring stride
constexpr int DR_META = 8;                        // tile-offset registers per lane, 64 tiles each
constexpr int DR_MAX_TPW = 64 * DR_META - 15;     // tiles one wave can own (from its first chunk's start)
constexpr int DR_CUS = 256;                       // workgroups per launch: one per CU of the MI355X

struct RingSmem {
    uint8_t* ring;    // [wave][K, V][DR_RS]; after the tiles: comb [wave][16][DC_CROW] f32
    float* comb;
    u32x4* qf;        // [row tile][4 steps][hi, lo][64] rotated query fragments (coded tiles)
    u32x4* kmask;     // [9]
    float* cm;        // [8][16]
    float* cl;        // [8][16]
    float* mrow;      // [coded, exact][16]
    float* lrow;      // [coded, exact][16]
};
constexpr int DR_QF = 4 * 2 * 64;                 // u32x4 per row tile's fragments (8 KB)
template <int RT>
__device__ __forceinline__ RingSmem ring_carve(uint8_t* smem) {
    RingSmem s;
    uint8_t* b = smem;
    s.ring = b; b += (size_t)DR_WAVES * 2 * DR_RS;
    s.comb = reinterpret_cast<float*>(s.ring);
    s.qf = reinterpret_cast<u32x4*>(b); b += (size_t)RT * DR_QF * 16;
    s.kmask = reinterpret_cast<u32x4*>(b); b += 9 * 16;
    float* f = reinterpret_cast<float*>(b);
    s.cm = f; f += DR_WAVES * 16;
    s.cl = f; f += DR_WAVES * 16;
    s.mrow = f; f += 32;
    s.lrow = f;
    return s;
}
template <int RT>
constexpr size_t dr_smem() { return (size_t)DR_WAVES * 2 * DR_RS + (size_t)RT * DR_QF * 16 + 9 * 16 + (2 * DR_WAVES * 16 + 64) * 4; }
static_assert(DR_WAVES * 16 * DC_CROW * 4 <= DR_WAVES * 2 * DR_RS, "combine rows fit in the rings");
static_assert(dr_smem<2>() <= 160 * 1024, "one workgroup per CU");

// 8 consecutive bf16 at ring element a (any 2-byte alignment, a may run past the ring's
// end): the dword indices are taken modulo the ring.
__device__ __forceinline__ u32x4 lds_row8_wrap(const uint32_t* w, int a) {
    constexpr int M = DR_RING / 4 - 1;
    const int w0 = a >> 1;
    const uint32_t sh = (uint32_t)(a & 1) * 16u;
    const uint32_t d0 = w[w0 & M], d1 = w[(w0 + 1) & M], d2 = w[(w0 + 2) & M], d3 = w[(w0 + 3) & M],
                   d4 = w[(w0 + 4) & M];
    return u32x4{__builtin_amdgcn_alignbit(d1, d0, sh), __builtin_amdgcn_alignbit(d2, d1, sh),
                 __builtin_amdgcn_alignbit(d3, d2, sh), __builtin_amdgcn_alignbit(d4, d3, sh)};
}

// Online softmax of the ring kernel, in log2 units (the query fragments carry log2(e) /
// sqrt(d)).  Each lane's reference m_run (its query row's) starts every score MFMA as the
// accumulator's initial value, so the MFMA returns score - reference directly.  The reference
// moves lazily: only when some score exceeds it by more than 8 (every weight then stays below
// 2^8), found from the lane's own scores; the cross-lane maximum of the row is taken only
// then, and on the wave's first tile (first: the sums and accumulators are still zero, so
// nothing is rescaled).  Returns through sv the scores relative to the (possibly moved)
// reference.
template <int NV, int SET>
__device__ __forceinline__ void ring_softmax_ref(float (&sv)[NV], bool& first, float& m_run, float& l_part) {
    float lmax = sv[0];
#pragma unroll
    for (int v = 1; v < NV; ++v) lmax = fmaxf(lmax, sv[v]);
    if (first || __builtin_amdgcn_ballot_w64(lmax > 8.f) != 0) {
        const float t = xmax32(xmax16(lmax));        // the row's maximum, relative
        const float shift = first ? t : (t > 8.f ? t : 0.f);
        if (!first) {
            const float alpha = __builtin_amdgcn_exp2f(-shift);
            l_part *= alpha;
            accs_scale<SET>(alpha);
        }
        m_run += shift;
#pragma unroll
        for (int v = 0; v < NV; ++v) sv[v] -= shift;
        first = false;
    }
}

// Softmax and value product of one tile for row tile R of the wave (accumulator set R):
// scores relative to the row tile's reference in sc.
template <int R, int NB>
__device__ __forceinline__ void ring_finish(f32x4 sc, const u32x2 (&vh)[NB], bool partial, int i0, int T, int grp,
                                            bool& first, float& m_run, float& l_part) {
    float sv[4] = {sc[0], sc[1], sc[2], sc[3]};
    if (partial) {
#pragma unroll
        for (int v = 0; v < 4; ++v) sv[v] = i0 + 4 * grp + v < T ? sv[v] : -INFINITY;
    }
    ring_softmax_ref<4, R>(sv, first, m_run, l_part);
    float pv[4];
#pragma unroll
    for (int v = 0; v < 4; ++v) pv[v] = __builtin_amdgcn_exp2f(sv[v]);
    l_part += (pv[0] + pv[1]) + (pv[2] + pv[3]);
    const u32x2 ph = {cvt_bf16x2(pv[0], pv[1]), cvt_bf16x2(pv[2], pv[3])};
    accs_mfma_bf16<R, NB>(vh, ph);
}

// One tile from a wave's ring (bf16): the arithmetic of tile_step, with the tile at ring
// element rb and the query fragments in registers, for each of the wave's RT row tiles (the
// K and V gathers are shared; each row tile has its own scores, softmax state and
// accumulator set).  Coded tiles: K rows m elements apart, V coordinate-major; WRAP gathers
// modulo the ring.  Exact tiles: rows of 128 (never wrapped: 4 KB tiles from a 4 KB-aligned
// start).
template <bool EXACT, bool WRAP, int KS, int NB, int RT>
__device__ __forceinline__ void ring_tile(int rb, int m, int i0, int T, bool partial, const uint16_t* rK,
                                          const uint16_t* rV, const u32x4 (&qfr)[RT][4][2], const u32x4* kmask,
                                          int col, int grp, bool (&first)[RT], float (&m_run)[RT],
                                          float (&l_part)[RT]) {
    u32x2 vh[NB];
    auto gather_v = [&]() {
#pragma unroll
        for (int b = 0; b < NB; ++b) {
            const int j = 16 * b + col;
            if constexpr (EXACT) {
                // rows past the exact slots in use hold no data: masked
                us2 h[2];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int a = i0 + 4 * grp + e < T ? rb + (4 * grp + e) * D + j : DR_RING_E;
                    h[e >> 1][e & 1] = rV[a];
                }
                vh[b] = u32x2{__builtin_bit_cast(uint32_t, h[0]), __builtin_bit_cast(uint32_t, h[1])};
            } else {
                // four consecutive positions at coordinate j (8-byte aligned, so never split by
                // the ring's end); past the tile's size: the zeros after the ring
                int a = rb + 16 * j + 4 * grp;
                if constexpr (WRAP) a &= DR_RING_E - 1;
                a = j < m ? a : DR_RING_E;
                vh[b] = *reinterpret_cast<const u32x2*>(rV + a);
            }
        }
    };
    if constexpr (KS < 4) gather_v();
    const uint32_t* rK32 = reinterpret_cast<const uint32_t*>(rK);
    f32x4 sc[RT];
#pragma unroll
    for (int r = 0; r < RT; ++r) sc[r] = f32x4{-m_run[r], -m_run[r], -m_run[r], -m_run[r]};
#pragma unroll
    for (int s = 0; s < KS; ++s) {
        if (KS >= 4 && s == 2) __builtin_amdgcn_sched_barrier(0);
        const int c0 = 32 * s + 8 * grp;
        const int mm = EXACT ? D : m;
        int nv = mm - c0;
        nv = nv < 0 ? 0 : (nv > 8 ? 8 : nv);
        const int a = rb + (int)__umul24((uint32_t)col, (uint32_t)mm) + c0;
        const u32x4 kh = (WRAP ? lds_row8_wrap(rK32, a) : lds_row8_bf16(rK32, a)) & kmask[nv];
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            sc[r] = mfma(kh, qfr[r][s][0], sc[r]);
            sc[r] = mfma(kh, qfr[r][s][1], sc[r]);
        }
    }
    if constexpr (KS >= 4) {
        __builtin_amdgcn_sched_barrier(0);
        gather_v();
    }
    ring_finish<0, NB>(sc[0], vh, partial, i0, T, grp, first[0], m_run[0], l_part[0]);
    if constexpr (RT == 2) ring_finish<1, NB>(sc[RT - 1], vh, partial, i0, T, grp, first[RT - 1], m_run[RT - 1], l_part[RT - 1]);
}

// Softmax and value products of a pair of small tiles for row tile R (accumulator set R).
template <int R>
__device__ __forceinline__ void ring_pair_finish(f32x4 sA, f32x4 sB, const u32x2 (&va)[2], const u32x2 (&vb)[2],
                                                 bool& first, float& m_run, float& l_part) {
    float sv[8] = {sA[0], sA[1], sA[2], sA[3], sB[0], sB[1], sB[2], sB[3]};
    ring_softmax_ref<8, R>(sv, first, m_run, l_part);
    float pv[8];
#pragma unroll
    for (int v = 0; v < 8; ++v) pv[v] = __builtin_amdgcn_exp2f(sv[v]);
    l_part += ((pv[0] + pv[1]) + (pv[2] + pv[3])) + ((pv[4] + pv[5]) + (pv[6] + pv[7]));
    const u32x2 pha = {cvt_bf16x2(pv[0], pv[1]), cvt_bf16x2(pv[2], pv[3])};
    const u32x2 phb = {cvt_bf16x2(pv[4], pv[5]), cvt_bf16x2(pv[6], pv[7])};
    accs_mfma_bf16<R, 2>(va, pha);
    accs_mfma_bf16<R, 2>(vb, phb);
}

// Two consecutive small tiles (sizes <= 32, neither wrapped nor ragged) in one step: their
// gathers and MFMA chains interleave, and they share one reference test and the loop's
// bookkeeping.
template <int RT>
__device__ __forceinline__ void ring_pair(int rbA, int mA, int rbB, int mB, const uint16_t* rK, const uint16_t* rV,
                                          const u32x4 (&qfr)[RT][4][2], const u32x4* kmask, int col, int grp,
                                          bool (&first)[RT], float (&m_run)[RT], float (&l_part)[RT]) {
    const uint32_t* rK32 = reinterpret_cast<const uint32_t*>(rK);
    u32x2 va[2], vb[2];
#pragma unroll
    for (int b = 0; b < 2; ++b) {
        const int j = 16 * b + col;
        const int aa = j < mA ? rbA + 16 * j + 4 * grp : DR_RING_E;
        const int ab = j < mB ? rbB + 16 * j + 4 * grp : DR_RING_E;
        va[b] = *reinterpret_cast<const u32x2*>(rV + aa);
        vb[b] = *reinterpret_cast<const u32x2*>(rV + ab);
    }
    int nvA = mA - 8 * grp, nvB = mB - 8 * grp;
    nvA = nvA < 0 ? 0 : (nvA > 8 ? 8 : nvA);
    nvB = nvB < 0 ? 0 : (nvB > 8 ? 8 : nvB);
    const u32x4 kA = lds_row8_bf16(rK32, rbA + (int)__umul24((uint32_t)col, (uint32_t)mA) + 8 * grp) & kmask[nvA];
    const u32x4 kB = lds_row8_bf16(rK32, rbB + (int)__umul24((uint32_t)col, (uint32_t)mB) + 8 * grp) & kmask[nvB];
    f32x4 sA[RT], sB[RT];
#pragma unroll
    for (int r = 0; r < RT; ++r) {
        const f32x4 minit = {-m_run[r], -m_run[r], -m_run[r], -m_run[r]};
        sA[r] = mfma(kA, qfr[r][0][0], minit);
        sB[r] = mfma(kB, qfr[r][0][0], minit);
        sA[r] = mfma(kA, qfr[r][0][1], sA[r]);
        sB[r] = mfma(kB, qfr[r][0][1], sB[r]);
    }
    ring_pair_finish<0>(sA[0], sB[0], va, vb, first[0], m_run[0], l_part[0]);
    if constexpr (RT == 2) ring_pair_finish<1>(sA[RT - 1], sB[RT - 1], va, vb, first[RT - 1], m_run[RT - 1], l_part[RT - 1]);
}

// ---- 5. combine of row tile R (accumulator set R): the coded waves into record 1 + j, the
//         exact waves into record 0, each in wave order (log2 units here; the records hold the
//         maxima in natural-log units, as the merge reads them).  Lane (col, grp) holds query
//         row col.  upair: the (sequence, KV head, row-tile group) unit of the workgroup.
template <int R, int RT>
__device__ __forceinline__ void combine_records(const DecParams& p, const RingSmem& sm, int upair, int nqp, int j,
                                                bool lastwg, int nxw, bool xw, int wave, int lane, int tid,
                                                int col, int grp, bool first, float m_run, float l_part) {
    const int sq = upair / (p.G * nqp), gq = upair % (p.G * nqp);
    const int g = gq / nqp, qt = RT * (gq % nqp) + R;
    if (qt >= p.nqt) return;            // (the whole workgroup: a group's second row tile past the last)
    const int unit = (sq * p.G + g) * p.nqt + qt;
    const int rows = min(16, p.rows_total - 16 * qt);
    const int nr4 = (rows + 3) & ~3;
    if (first) m_run = -INFINITY;       // no tile: an empty partial
    f32x4 acc[8];
    accs_read<R>(acc);
    const float lsum = xsum32(xsum16(l_part));
    if (lane < 16) { sm.cm[wave * 16 + col] = m_run; sm.cl[wave * 16 + col] = lsum; }
    __syncthreads();   // also: every wave is done with its ring, which comb reuses
    const int wc = DR_WAVES - nxw;
    if (tid < 32) {
        // every wave's entries are read at once (fixed trip count, waves outside [w_lo, w_hi)
        // predicated off), then folded in wave order
        const int r = tid & 15;
        const int w_lo = tid >= 16 ? wc : 0, w_hi = tid >= 16 ? DR_WAVES : wc;
        float mw[DR_WAVES], lw[DR_WAVES];
#pragma unroll
        for (int w = 0; w < DR_WAVES; ++w) {
            mw[w] = sm.cm[w * 16 + r];
            lw[w] = sm.cl[w * 16 + r];
        }
        float M = -INFINITY;
#pragma unroll
        for (int w = 0; w < DR_WAVES; ++w) M = w >= w_lo && w < w_hi ? fmaxf(M, mw[w]) : M;
        float Ls = 0.f;
#pragma unroll
        for (int w = 0; w < DR_WAVES; ++w)
            if (w >= w_lo && w < w_hi) Ls += mw[w] == -INFINITY ? 0.f : lw[w] * __builtin_amdgcn_exp2f(mw[w] - M);
        sm.mrow[tid] = M;
        sm.lrow[tid] = Ls;
    }
    __syncthreads();
    {
        const float mref = sm.mrow[(xw ? 16 : 0) + col];
        const float fac = m_run == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_run - mref);
        if (col < nr4) {
#pragma unroll
            for (int b = 0; b < 8; ++b)
                *reinterpret_cast<f32x4*>(&sm.comb[(wave * 16 + col) * DC_CROW + 16 * b + 4 * grp]) = acc[b] * fac;
        }
    }
    __syncthreads();
    float* recs = p.part + (int64_t)unit * p.nrec * DC_REC;
    const int n4 = nr4 * D / 4;
    for (int part = 0; part < (lastwg ? 2 : 1); ++part) {
        float* rec = recs + (int64_t)(part ? 0 : 1 + j) * DC_REC;
        const int w_lo = part ? wc : 0, w_hi = part ? DR_WAVES : wc;
        for (int idx = tid; idx < n4; idx += DR_THREADS) {
            const int ci = (idx >> 5) * DC_CROW + 4 * (idx & 31);   // row idx/32, float4 idx%32
            f32x4 cw[DR_WAVES];
#pragma unroll
            for (int w = 0; w < DR_WAVES; ++w) cw[w] = *reinterpret_cast<const f32x4*>(sm.comb + w * 16 * DC_CROW + ci);
            f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int w = 0; w < DR_WAVES; ++w)
                if (w >= w_lo && w < w_hi) s += cw[w];
            reinterpret_cast<f32x4*>(rec + 32)[idx] = s;
        }
        if (tid < 16) {
            rec[tid] = sm.mrow[16 * part + tid] * 0.6931471805599453f;   // ln 2: log2 -> natural units
            rec[16 + tid] = sm.lrow[16 * part + tid];
        }
    }
}

// RT = 2: every wave serves two row tiles of the same (sequence, KV head) (a batch of query
// rows): the ring, the K and V gathers and the loop's bookkeeping are shared, the scores,
// softmax states, accumulator sets (a0..a31, a32..a63) and records are the row tiles' own.
template <int RT>
__global__ __launch_bounds__(DR_THREADS, 1) void decode_ring_kernel(DecParams p) {
    extern __shared__ __attribute__((aligned(16))) uint8_t smem[];
    const int nqp = (p.nqt + RT - 1) / RT;       // groups of RT row tiles
    const int U = p.units / p.nqt * nqp;          // (sequence, KV head, row-tile group) units
    const int L = blockIdx.x;
    // workgroup j of the unit.  Workgroup L runs on XCD L mod 8: with a grid of a multiple of 8
    // workgroups, XCD x takes the x-th eighth of the unit-major order, so a unit's workgroups,
    // and the units of one KV head (the row tiles of a batch of queries, which stream the same
    // coefficients), share one L2.  For one sequence of 8 KV heads this is unit = L mod 8.
    int unit, j;
    if ((gridDim.x & 7) == 0) {
        const int Lp = (L & 7) * (int)(gridDim.x >> 3) + (L >> 3);
        unit = Lp / p.wpu;
        j = Lp % p.wpu;
    } else {
        unit = L % U;
        j = L / U;
    }
    const int sq = unit / (p.G * nqp), gq = unit % (p.G * nqp);
    const int g = gq / nqp, qp = gq % nqp;
    const DecSeq& S = p.seq[sq];
    const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
    const int lane = lane_now(), tid = 64 * wave + lane, grp = lane >> 4, col = lane & 15;
    RingSmem sm = ring_carve<RT>(smem);
    const float qscale = 0.12751743082459868f;  // log2(e) / sqrt(128)
    const bool lastwg = j == p.wpu - 1;
    const int nxw = lastwg ? p.n_xw : 0;          // exact waves of this workgroup (its last ones)
    const bool xw = wave >= DR_WAVES - nxw;
    const int ncw = DR_WAVES * p.wpu - p.n_xw;   // coded waves of the unit
    const int T = p.total_tiles;
    const int nexact = (int)S.n_exact;
    int t0, t1;
    if (!xw) {
        const int k = DR_WAVES * j + wave;
        t0 = (int)((int64_t)k * T / ncw);
        t1 = (int)((int64_t)(k + 1) * T / ncw);
    } else {
        const int xi = wave - (DR_WAVES - nxw);
        const int X = (nexact + 15) >> 4;
        t0 = xi * X / nxw;
        t1 = (xi + 1) * X / nxw;
    }
    t0 = __builtin_amdgcn_readfirstlane(t0);
    t1 = __builtin_amdgcn_readfirstlane(t1);

    // ---- 1. loads of the prologue, in this order: the first rank of every tile from the start
    //         of this wave's first chunk to its last tile and the chunk bases (coded waves; 16
    //         loads), then the basis rows 16 wave .. 16 wave + 15 and the query rows (8 + 4 RT
    //         loads: every wave rotates its 16 directions of q' for the whole workgroup).  They are
    //         issued in asm and waited for by load count: the metadata once the basis is the only
    //         younger load, the basis once only the ring loads issued after it are younger.
    //         Every lane loads a valid address; values of lanes outside the range are dropped.
    const int c0 = t0 >> 4;
    uint32_t mr[DR_META], cbr[DR_META];
#pragma unroll
    for (int b = 0; b < DR_META; ++b) {
        const int tt = 16 * c0 + 64 * b + lane;
        const bool in = !xw && tt < t1;
        const uint8_t* ap = in ? S.srank + (int64_t)tt * 16 : S.srank;
        const uint32_t* cp = in ? S.chunk_off + c0 + 4 * b + (lane >> 4) : S.chunk_off;
        asm volatile("global_load_ubyte %0, %1, off" : "=v"(mr[b]) : "v"(ap) : "memory");
        asm volatile("global_load_dword %0, %1, off" : "=v"(cbr[b]) : "v"(cp) : "memory");
    }
    const uint16_t* qsrc = reinterpret_cast<const uint16_t*>(S.q);
    const float* P = p.PK + (int64_t)g * D * D;
    bool q_ok[RT];
    u32x4 pa[4][2], qr[RT][4];
#pragma unroll
    for (int r = 0; r < RT; ++r) {
        const int qrow_l = 16 * (RT * qp + r) + col;
        q_ok[r] = qrow_l < p.rows_total;
    }
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        const float* src = P + (16 * wave + col) * D + 32 * s + 8 * grp;
        asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(pa[s][0]) : "v"(src) : "memory");
        asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(pa[s][1]) : "v"(src + 4) : "memory");
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            const int qrow_l = 16 * (RT * qp + r) + col;
            const int query_l = q_ok[r] ? qrow_l / p.hpg : 0, hh_l = q_ok[r] ? qrow_l % p.hpg : 0;
            // 2-byte aligned: gfx950 serves it whole
            const uint16_t* qs = qsrc + ((int64_t)query_l * p.H + g * p.hpg + hh_l) * D + 32 * s + 8 * grp;
            asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(qr[r][s]) : "v"(qs) : "memory");
        }
    }
    static_assert(DR_META == 8, "the waits below name every metadata register");
    if constexpr (RT == 1)
        asm volatile("s_waitcnt vmcnt(12)" : "+v"(mr[0]), "+v"(mr[1]), "+v"(mr[2]), "+v"(mr[3]), "+v"(mr[4]), "+v"(mr[5]),
                     "+v"(mr[6]), "+v"(mr[7]), "+v"(cbr[0]), "+v"(cbr[1]), "+v"(cbr[2]), "+v"(cbr[3]), "+v"(cbr[4]),
                     "+v"(cbr[5]), "+v"(cbr[6]), "+v"(cbr[7]) :: "memory");
    else
        asm volatile("s_waitcnt vmcnt(16)" : "+v"(mr[0]), "+v"(mr[1]), "+v"(mr[2]), "+v"(mr[3]), "+v"(mr[4]), "+v"(mr[5]),
                     "+v"(mr[6]), "+v"(mr[7]), "+v"(cbr[0]), "+v"(cbr[1]), "+v"(cbr[2]), "+v"(cbr[3]), "+v"(cbr[4]),
                     "+v"(cbr[5]), "+v"(cbr[6]), "+v"(cbr[7]) :: "memory");
#pragma unroll
    for (int b = 0; b < DR_META; ++b) {
        const int tt = 16 * c0 + 64 * b + lane;
        const bool in = !xw && tt < t1;
        mr[b] = in ? mr[b] : 0u;
        cbr[b] = in ? cbr[b] : 0u;
    }
    // lane i of register b: tile 16 c0 + 64 b + i (chunk c0 + 4 b + i / 16, one DPP row per
    // chunk): element offset in the head stream = chunk base + sizes of the chunk's earlier tiles
    uint32_t off[DR_META];
#pragma unroll
    for (int b = 0; b < DR_META; ++b) {
        const uint32_t units = 16u * mr[b];
        off[b] = cbr[b] + row_scan16(units) - units;
    }
    // the wave's element range of its stream
    uint32_t e0, e1;
    if (xw) {
        e0 = 16u * D * (uint32_t)t0;
        e1 = (uint32_t)min(16 * t1, nexact) * D;
    } else if (t1 > t0) {
        e0 = (uint32_t)__builtin_amdgcn_readlane((int)off[0], t0 & 15);
        // the last tile's offset and size: read from every block, kept from block il / 64 (no
        // register is picked by a run-time index, which would go through scratch memory)
        const int il = t1 - 1 - 16 * c0;
        const int nb = il >> 6;
        uint32_t ol = 0u, ml = 0u;
#pragma unroll
        for (int b = 0; b < DR_META; ++b) {
            const uint32_t ob = (uint32_t)__builtin_amdgcn_readlane((int)off[b], il & 63);
            const uint32_t mb = (uint32_t)__builtin_amdgcn_readlane((int)mr[b], il & 63);
            ol = nb == b ? ob : ol;
            ml = nb == b ? mb : ml;
        }
        e1 = ol + 16u * ml;
    } else {
        e0 = e1 = 0;
    }
    e0 = __builtin_amdgcn_readfirstlane(e0);
    e1 = __builtin_amdgcn_readfirstlane(e1);

    // ---- 2. ring loads: unit u = bytes [base + 1 KB u, + 1 KB) of the wave's range (lanes past
    //         its end masked), into ring slot u mod 8 of K and of V; two loads per unit.  The
    //         first 8 units go out now; a range of fewer units is padded with one-lane loads of
    //         its first bytes into the slots it leaves unused, so exactly 16 ring loads are
    //         younger than the basis when it is waited for.  The coefficients are read once per
    //         call, so the loads carry the non-temporal hint: their lines leave L2 first, and the
    //         small data every call reuses (bases, ranks, chunk table, records) stays there.
    uint8_t* rK = sm.ring + (size_t)wave * 2 * DR_RS;
    uint8_t* rV = rK + DR_RS;
    const int64_t hoff = xw ? (int64_t)g * p.cap * D : (int64_t)g * p.coef_stride;
    const uint8_t* kg = reinterpret_cast<const uint8_t*>(xw ? S.k_exact : S.coef_k) + hoff * 2;
    const uint8_t* vg = reinterpret_cast<const uint8_t*>(xw ? S.v_exact : S.coef_v) + hoff * 2;
    const uint32_t base = (2u * e0) & ~15u;
    const uint32_t eb = 2u * e1;
    const int n_units = e1 > e0 ? (int)((eb - base + DR_UNIT - 1) / DR_UNIT) : 0;
    const uint32_t ldsK = __builtin_amdgcn_readfirstlane((uint32_t)(size_t)(lds_u8*)rK);
    const uint32_t ldsV = __builtin_amdgcn_readfirstlane((uint32_t)(size_t)(lds_u8*)rV);
    const uint32_t lane16 = 16u * (uint32_t)lane;
    auto issue = [&](int u) {
        const uint32_t o = base + (uint32_t)u * DR_UNIT + lane16;
        const uint32_t sl = (uint32_t)(u & (DR_NU - 1)) * DR_UNIT;
        if (o < eb) {     // lane 0 always is: unit u < n_units starts before the range's end
            asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
                         :: "v"(kg + o), "s"(ldsK + sl) : "memory", "m0");
            asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
                         :: "v"(vg + o), "s"(ldsV + sl) : "memory", "m0");
        }
    };
    int u_iss = n_units < DR_NU ? n_units : DR_NU;
    for (int u = 0; u < DR_NU; ++u) {
        if (u < u_iss) {
            issue(u);
        } else if (lane == 0) {
            const uint32_t sl = (uint32_t)u * DR_UNIT;
            asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
                         :: "v"(kg + base), "s"(ldsK + sl) : "memory", "m0");
            asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
                         :: "v"(vg + base), "s"(ldsV + sl) : "memory", "m0");
        }
    }
    asm volatile("s_waitcnt vmcnt(16)" : "+v"(pa[0][0]), "+v"(pa[0][1]), "+v"(pa[1][0]), "+v"(pa[1][1]),
                 "+v"(pa[2][0]), "+v"(pa[2][1]), "+v"(pa[3][0]), "+v"(pa[3][1]), "+v"(qr[0][0]), "+v"(qr[0][1]),
                 "+v"(qr[0][2]), "+v"(qr[0][3]) :: "memory");
    if constexpr (RT == 2)      // (already landed: the wait above covers every older load)
        asm volatile("" : "+v"(qr[RT - 1][0]), "+v"(qr[RT - 1][1]), "+v"(qr[RT - 1][2]), "+v"(qr[RT - 1][3]) :: "memory");

    // ---- 3. while the ring fills: q' = P_K q log2(e) / sqrt(d) by MFMA (C lane -> query row
    //         col, directions 16 wave + 4 grp + v) into the score fragments, for each row tile;
    //         the V rings' zero pads and the K-row masks.  Then every coded wave keeps its
    //         fragments in registers; the exact waves form theirs from q itself, which every
    //         wave holds in the fragment layout.
    {
        f32x4 c[RT];
#pragma unroll
        for (int r = 0; r < RT; ++r) c[r] = f32x4{0, 0, 0, 0};
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            float a8[8];
#pragma unroll
            for (int e = 0; e < 4; ++e) { a8[e] = __uint_as_float(pa[s][0][e]); a8[4 + e] = __uint_as_float(pa[s][1][e]); }
            u32x4 ah, al;
            split8(a8, ah, al);
#pragma unroll
            for (int r = 0; r < RT; ++r) {
                const u32x4 qb = q_ok[r] ? qr[r][s] : u32x4{0, 0, 0, 0};
                c[r] = mfma(ah, qb, c[r]);
                c[r] = mfma(al, qb, c[r]);
            }
        }
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            uint32_t h[4], l[4];
#pragma unroll
            for (int v = 0; v < 4; ++v) split_bf16(c[r][v] * qscale, h[v], l[v]);
            uint32_t* qf32 = reinterpret_cast<uint32_t*>(sm.qf + r * DR_QF);
            const int s = wave >> 1, gp = 2 * (wave & 1) + (grp >> 1), dw = 2 * (grp & 1);
            *reinterpret_cast<u32x2*>(qf32 + ((s * 2 + 0) * 64 + gp * 16 + col) * 4 + dw) = u32x2{pack2(h[0], h[1]), pack2(h[2], h[3])};
            *reinterpret_cast<u32x2*>(qf32 + ((s * 2 + 1) * 64 + gp * 16 + col) * 4 + dw) = u32x2{pack2(l[0], l[1]), pack2(l[2], l[3])};
        }
    }
    if (lane < DR_PAD / 4) reinterpret_cast<uint32_t*>(rV + DR_RING)[lane] = 0u;
    if (tid >= 64 && tid < 64 + 9) {
        const int nv = tid - 64;
        u32x4 mk;
#pragma unroll
        for (int k = 0; k < 4; ++k) mk[k] = nv >= 2 * k + 2 ? 0xFFFFFFFFu : (nv == 2 * k + 1 ? 0x0000FFFFu : 0u);
        sm.kmask[nv] = mk;
    }
    __syncthreads();
    u32x4 qfr[RT][4][2];
    if (!xw) {
#pragma unroll
        for (int r = 0; r < RT; ++r)
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                qfr[r][s][0] = sm.qf[r * DR_QF + (s * 2) * 64 + lane];
                qfr[r][s][1] = sm.qf[r * DR_QF + (s * 2 + 1) * 64 + lane];
            }
    } else {
        // the exact rows' fragments: q itself (lane: query row col, elements 32 s + 8 grp ..)
#pragma unroll
        for (int r = 0; r < RT; ++r)
#pragma unroll
            for (int s = 0; s < 4; ++s) {
                float v8[8];
#pragma unroll
                for (int e = 0; e < 8; ++e) {
                    const float val = (e & 1) ? bf_hi(qr[r][s][e >> 1]) : bf_lo(qr[r][s][e >> 1]);
                    v8[e] = q_ok[r] ? val * qscale : 0.f;
                }
                split8(v8, qfr[r][s][0], qfr[r][s][1]);
            }
    }
    // allow n units (2 n loads) in flight, n rounded down to even: at most one unit more is
    // waited for than the tile needs (and the padding loads of a short range, which are younger
    // than all of its units)
    auto wait_units = [&](int n) {
        if (n < 4) {
            if (n < 2) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
            else asm volatile("s_waitcnt vmcnt(4)" ::: "memory");
        } else {
            if (n < 6) asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
            else asm volatile("s_waitcnt vmcnt(12)" ::: "memory");
        }
    };
    // before a tile: load every unit up to 8 past its first one (their slots hold units no
    // remaining tile needs), then wait for the units it spans
    auto land = [&](uint32_t bs, uint32_t tbytes) {
        const int first_u = (int)(bs >> 10);
        const int u_lim = n_units < first_u + DR_NU ? n_units : first_u + DR_NU;
        while (u_iss < u_lim) {
            issue(u_iss);
            ++u_iss;
        }
        if (tbytes) wait_units(u_iss - (int)((bs + tbytes - 1) >> 10) - 1);
    };

    // ---- 4. tiles
    float m_run[RT], l_part[RT];        // the reference is set on the first tile
    bool first[RT];
#pragma unroll
    for (int r = 0; r < RT; ++r) { m_run[r] = 0.f; l_part[r] = 0.f; first[r] = true; }
    accs_zero<0>();
    if constexpr (RT == 2) accs_zero<RT - 1>();
    const uint16_t* rK16 = reinterpret_cast<const uint16_t*>(rK);
    const uint16_t* rV16 = reinterpret_cast<const uint16_t*>(rV);
    if (xw) {
        for (int t = t0; t < t1; ++t) {
            const uint32_t bs = 2u * 16u * D * (uint32_t)t - base;
            land(bs, 2u * 16u * D);
            const int rb = (int)((bs & (DR_RING - 1)) >> 1);
            ring_tile<true, false, 4, 8, RT>(rb, D, 16 * t, nexact, 16 * t + 16 > nexact, rK16, rV16, qfr, sm.kmask,
                                             col, grp, first, m_run, l_part);
        }
    } else {
        // the head's last tile is the only one with fewer than 16 positions
        const int t_part = (p.N & 15) ? T - 1 : -1;
        // block b's offsets and sizes are always read from off[0] / mr[0]: the blocks shift
        // down by one after each
        for (int b = 0; b < DR_META; ++b) {
            const int lo = max(t0, 16 * c0 + 64 * b), hi = min(t1, 16 * c0 + 64 * b + 64);
            if (lo >= hi) break;
            const uint32_t co = off[0], cmk = mr[0];
#pragma unroll
            for (int k = 0; k + 1 < DR_META; ++k) {
                off[k] = off[k + 1];
                mr[k] = mr[k + 1];
            }
            for (int t = lo; t < hi;) {
                const int li = (t - 16 * c0) & 63;
                const uint32_t tb = (uint32_t)__builtin_amdgcn_readlane((int)co, li);
                const int mi = __builtin_amdgcn_readlane((int)cmk, li);
                const uint32_t bs = 2u * tb - base;           // byte offset from the ring's origin
                const int rb = (int)((bs & (DR_RING - 1)) >> 1);
                const bool wrap = rb + 16 * mi > DR_RING_E;
                const bool small = mi <= 32 && !wrap && t != t_part;
                if (small && t + 1 < hi) {
                    // the next tile follows this one in the stream
                    const int mj = __builtin_amdgcn_readlane((int)cmk, li + 1);
                    const int rb2 = (int)(((bs + 32u * (uint32_t)mi) & (DR_RING - 1)) >> 1);
                    if (mj <= 32 && rb2 + 16 * mj <= DR_RING_E && t + 1 != t_part) {
                        land(bs, 32u * (uint32_t)(mi + mj));
                        ring_pair<RT>(rb, mi, rb2, mj, rK16, rV16, qfr, sm.kmask, col, grp, first, m_run, l_part);
                        t += 2;
                        continue;
                    }
                }
                land(bs, 32u * (uint32_t)mi);
                if (small) {
                    ring_tile<false, false, 1, 2, RT>(rb, mi, 0, CHUNK, false, rK16, rV16, qfr, sm.kmask, col, grp, first, m_run, l_part);
                } else {
                    const int i0 = 16 * (t & 15);
                    const int64_t ct = (int64_t)(t >> 4) * CHUNK;
                    const int Tc = (int)(p.N - ct < CHUNK ? p.N - ct : CHUNK);
                    const bool partial = t == t_part;
                    if (!wrap) {
                        if (mi <= 32) ring_tile<false, false, 1, 2, RT>(rb, mi, i0, Tc, partial, rK16, rV16, qfr, sm.kmask, col, grp, first, m_run, l_part);
                        else if (mi <= 64) ring_tile<false, false, 2, 4, RT>(rb, mi, i0, Tc, partial, rK16, rV16, qfr, sm.kmask, col, grp, first, m_run, l_part);
                        else ring_tile<false, false, 4, 8, RT>(rb, mi, i0, Tc, partial, rK16, rV16, qfr, sm.kmask, col, grp, first, m_run, l_part);
                    } else {
                        if (mi <= 32) ring_tile<false, true, 1, 2, RT>(rb, mi, i0, Tc, partial, rK16, rV16, qfr, sm.kmask, col, grp, first, m_run, l_part);
                        else if (mi <= 64) ring_tile<false, true, 2, 4, RT>(rb, mi, i0, Tc, partial, rK16, rV16, qfr, sm.kmask, col, grp, first, m_run, l_part);
                        else ring_tile<false, true, 4, 8, RT>(rb, mi, i0, Tc, partial, rK16, rV16, qfr, sm.kmask, col, grp, first, m_run, l_part);
                    }
                }
                ++t;
            }
        }
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    combine_records<0, RT>(p, sm, unit, nqp, j, lastwg, nxw, xw, wave, lane, tid, col, grp, first[0], m_run[0], l_part[0]);
    if constexpr (RT == 2) {
        __syncthreads();   // every wave is done with the first row tile's combine area
        combine_records<RT - 1, RT>(p, sm, unit, nqp, j, lastwg, nxw, xw, wave, lane, tid, col, grp, first[RT - 1],
                                    m_run[RT - 1], l_part[RT - 1]);
    }
}
// ----------------------------------------------------------------------------------------
// Merge of the partial records of one (sequence, KV head, row tile): log-sum-exp over the
// records (record 0 = exact slots, original space; records 1.. = coded tile ranges, rank
// space), back-rotation of the rank-space sum with P_V^T, division by the softmax
// denominator.  A separate launch: the kernel boundary publishes every record, so no
// workgroup of the streaming kernel needs a device-wide fence.
// The merge is spread over one workgroup per (unit, query row, block of 32 output columns),
// so no workgroup pulls more than one row of every record (512 bytes each) and a 128 x 32
// slab of the basis; every load is issued before the first wait, and the small per-row
// reductions are repeated by the column blocks instead of exchanged.
struct MergeParams {
    const float* part;
    const float* PV;
    void* out;              // [S][Q][H][d] of this launch's sequences
    int64_t out_seq_stride; // elements per sequence
    int G, H, hpg, nqt, rows_total, n_wg, rpu;
    int nrec;               // records per unit; those past n_wg + 1 are original-space (anchors)
    int xcd_m;              // > 0: XCD-aware order, each KV head's workgroups on 8 / G XCDs (G < 8)
                            // or head g on XCD g mod 8 (G a multiple of 8); 0: plain order
};

constexpr int MG_THREADS = 256;
constexpr int MG_COLS = 32;                       // output columns per workgroup
constexpr int MG_CB = D / MG_COLS;                // column blocks per row
constexpr int MG_RPT = 32;                        // coded records per thread in registers

template <bool F32>
__global__ __launch_bounds__(MG_THREADS) void decode_merge_kernel(MergeParams p) {
    typedef typename Elem<F32>::T ET;
    __shared__ float wr[DC_MAX_REC];              // record weights exp(m_r - M)
    __shared__ float red[2][MG_THREADS / 64];
    __shared__ float accR[2][D];
    __shared__ float part8[8][MG_COLS];
    // workgroup -> (unit, row, column block).  Workgroups are dispatched round-robin over the
    // 8 XCDs (workgroup L on XCD L mod 8), so the XCD-aware order puts every workgroup of KV
    // head g on the XCDs that ran g's streaming workgroups: the head's basis slabs and records
    // are then fetched into those XCDs' L2 only.
    const int P = p.rpu * MG_CB;                  // workgroups per unit
    const int units = p.G * p.nqt;
    const int nsq = (int)(gridDim.x / (P * units));
    int unit, wi;
    if (p.xcd_m > 0) {
        const int x = blockIdx.x & 7, k = blockIdx.x >> 3;
        const int per_head = nsq * p.nqt * P;    // workgroups of one KV head
        int gh, idx;
        if (p.G >= 8) {                           // heads x, x + 8, ...: k-th of them in order
            gh = x + 8 * (k / per_head);
            idx = k % per_head;
        } else {                                  // head x / m over m XCDs, interleaved
            gh = x / p.xcd_m;
            idx = k * p.xcd_m + x % p.xcd_m;
        }
        const int uh = idx / P;                   // (sequence, row tile) of the head
        wi = idx % P;
        unit = ((uh / p.nqt) * p.G + gh) * p.nqt + uh % p.nqt;
    } else {
        unit = blockIdx.x / P;
        wi = blockIdx.x % P;
    }
    const int cb = wi % MG_CB;
    const int row = wi / MG_CB;
    const int sq = unit / units, gq = unit % units;
    const int g = gq / p.nqt, qt = gq % p.nqt;
    const int rows = min(16, p.rows_total - 16 * qt);
    if (row >= rows) return;                      // row tiles with fewer rows (workgroup-uniform)
    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int nrec = p.nrec;
    const int nrc = p.n_wg + 1;                   // records 1 .. nrc - 1 are rank-space
    const float* recs = p.part + (int64_t)unit * nrec * DC_REC;

    // ---- 1. issue every load: this row's max and sum of each record, its rank-space row of
    //          the coded records (thread -> coordinate j, half h of the records), the basis
    //          slab rows 16 jg .. 16 jg + 15 at column c, and the exact record's row piece
    const int j = tid & (D - 1), h = tid >> 7;
    const int c = tid & (MG_COLS - 1), jg = tid >> 5;
    float ms[2], ls[2];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int r = tid + k * MG_THREADS;
        const int rr = r < nrec ? r : 0;
        ms[k] = recs[(int64_t)rr * DC_REC + row];
        ls[k] = recs[(int64_t)rr * DC_REC + 16 + row];
    }
    float a[MG_RPT];
#pragma unroll
    for (int u = 0; u < MG_RPT; ++u) {
        const int r = 1 + h + 2 * u;
        a[u] = r < nrc ? recs[(int64_t)r * DC_REC + 32 + row * D + j] : 0.f;
    }
    const float* PV = p.PV + (int64_t)g * D * D + MG_COLS * cb + c;
    float pb[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) pb[i] = PV[(int64_t)(16 * jg + i) * D];
    const float ex = tid < MG_COLS ? recs[32 + row * D + MG_COLS * cb + tid] : 0.f;

    // ---- 2. row maximum over the records, record weights, softmax denominator
    float mx = fmaxf(tid < nrec ? ms[0] : -INFINITY, tid + MG_THREADS < nrec ? ms[1] : -INFINITY);
    for (int r = tid + 2 * MG_THREADS; r < nrec; r += MG_THREADS) mx = fmaxf(mx, recs[(int64_t)r * DC_REC + row]);
    mx = xmax32(xmax16(wave_max16(mx)));
    if (lane == 0) red[0][wave] = mx;
    __syncthreads();
    float M = red[0][0];
#pragma unroll
    for (int w = 1; w < MG_THREADS / 64; ++w) M = fmaxf(M, red[0][w]);
    float lsum = 0.f;
#pragma unroll
    for (int k = 0; k < 2; ++k) {
        const int r = tid + k * MG_THREADS;
        if (r < nrec) {
            const float wgt = ms[k] == -INFINITY ? 0.f : fast_exp(ms[k] - M);
            wr[r] = wgt;
            lsum += wgt * ls[k];
        }
    }
    for (int r = tid + 2 * MG_THREADS; r < nrec; r += MG_THREADS) {
        const float m = recs[(int64_t)r * DC_REC + row];
        const float wgt = m == -INFINITY ? 0.f : fast_exp(m - M);
        wr[r] = wgt;
        lsum += wgt * recs[(int64_t)r * DC_REC + 16 + row];
    }
    // fixed-order sum: lanes, then waves
    lsum = xsum32(xsum16(lsum + shfl_xor_f(lsum, 1)));
    lsum += shfl_xor_f(lsum, 2);
    lsum += shfl_xor_f(lsum, 4);
    lsum += shfl_xor_f(lsum, 8);
    if (lane == 0) red[1][wave] = lsum;
    __syncthreads();
    float L = red[1][0];
#pragma unroll
    for (int w = 1; w < MG_THREADS / 64; ++w) L += red[1][w];

    // ---- 3. weighted sum of the coded records' rank-space rows (two halves, fixed order)
    float s = 0.f;
#pragma unroll
    for (int u = 0; u < MG_RPT; ++u) {
        const int r = 1 + h + 2 * u;
        s += (r < nrc ? wr[r] : 0.f) * a[u];
    }
    for (int r = 1 + h + 2 * MG_RPT; r < nrc; r += 2) s += wr[r] * recs[(int64_t)r * DC_REC + 32 + row * D + j];
    accR[h][j] = s;
    __syncthreads();

    // ---- 4. back-rotation: out[c] = sum_j accR[j] P_V[j][c], 8 groups of 16 coordinates
    float o = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) {
        const int jj = 16 * jg + i;
        o += (accR[0][jj] + accR[1][jj]) * pb[i];
    }
    part8[jg][c] = o;
    __syncthreads();
    if (tid < MG_COLS) {
        float t = part8[0][tid];
#pragma unroll
        for (int k = 1; k < 8; ++k) t += part8[k][tid];
        float e = wr[0] * ex;
        for (int r = nrc; r < nrec; ++r) e += wr[r] * recs[(int64_t)r * DC_REC + 32 + row * D + MG_COLS * cb + tid];
        const float val = (t + e) / L;
        const int qrow = 16 * qt + row;
        const int query = qrow / p.hpg, hh = qrow % p.hpg;
        ET* out = reinterpret_cast<ET*>(p.out) + (int64_t)sq * p.out_seq_stride;
        const int64_t oi = ((int64_t)query * p.H + g * p.hpg + hh) * D + MG_COLS * cb + tid;
        if constexpr (F32) out[oi] = val;
        else out[oi] = (uint16_t)f32_to_bf16(val);
    }
}
// The same merge for units with many query rows: one workgroup per (unit, block of 32 output
// columns) takes every row of the unit, so the basis slab is read once per unit and column
// block (into LDS) instead of once per row, and each record row is read by one thread.  The
// slab's loads and the records' go out in batches before their first use; the back-rotation
// of the 16 x 128 rank-space rows by the 128 x 32 slab runs as fp32 MFMAs (16x16x4, two waves,
// one 16-column tile each).  Fixed-order sums throughout.
template <bool F32>
__global__ __launch_bounds__(MG_THREADS) void decode_merge_rows_kernel(MergeParams p) {
    typedef typename Elem<F32>::T ET;
    __shared__ float wgt[16][DC_MAX_REC];          // record weights exp(m_r - M) per row
    __shared__ float Lr[16];
    __shared__ float accR[16][D + 1];
    __shared__ float slab[D][MG_COLS + 1];
    const int units = p.G * p.nqt;
    const int nsq = (int)(gridDim.x / (MG_CB * units));
    int unit, cb;
    if (p.xcd_m > 0) {
        const int x = blockIdx.x & 7, k = blockIdx.x >> 3;
        const int per_head = nsq * p.nqt * MG_CB;
        int gh, idx;
        if (p.G >= 8) {
            gh = x + 8 * (k / per_head);
            idx = k % per_head;
        } else {
            gh = x / p.xcd_m;
            idx = k * p.xcd_m + x % p.xcd_m;
        }
        const int uh = idx / MG_CB;
        cb = idx % MG_CB;
        unit = ((uh / p.nqt) * p.G + gh) * p.nqt + uh % p.nqt;
    } else {
        unit = blockIdx.x / MG_CB;
        cb = blockIdx.x % MG_CB;
    }
    const int sq = unit / units, gq = unit % units;
    const int g = gq / p.nqt, qt = gq % p.nqt;
    const int rows = min(16, p.rows_total - 16 * qt);
    const int tid = threadIdx.x;
    const int nrec = p.nrec;
    const int nrc = p.n_wg + 1;                   // records 1 .. nrc - 1 are rank-space
    const float* recs = p.part + (int64_t)unit * nrec * DC_REC;
    // 1. the basis slab rows j, columns 32 cb .. 32 cb + 31 (every load before the first store)
    const float* PV = p.PV + (int64_t)g * D * D + MG_COLS * cb;
    {
        constexpr int SPT = D * MG_COLS / MG_THREADS;
        float sv[SPT];
#pragma unroll
        for (int e = 0; e < SPT; ++e) {
            const int i = tid + e * MG_THREADS;
            sv[e] = PV[(int64_t)(i / MG_COLS) * D + i % MG_COLS];
        }
#pragma unroll
        for (int e = 0; e < SPT; ++e) {
            const int i = tid + e * MG_THREADS;
            slab[i / MG_COLS][i % MG_COLS] = sv[e];
        }
    }
    // the first (up to) four coded records' rows for step 3, requested ahead of step 2
    constexpr int EPT = 16 * D / MG_THREADS;
    const int nb0 = nrc - 1 < 4 ? nrc - 1 : 4;
    float x0[4][EPT];
#pragma unroll
    for (int k = 0; k < 4; ++k)
#pragma unroll
        for (int e = 0; e < EPT; ++e) {
            const int i = tid + e * MG_THREADS;
            x0[k][e] = recs[(int64_t)(1 + (k < nb0 ? k : 0)) * DC_REC + 32 + i];
        }
    // 2. per row: maximum over the records, weights, softmax denominator.  Thread (group q =
    //    tid / 16, row tid % 16) takes records q, q + 16, ..; the groups' maxima and sums are
    //    combined in group order.
    __shared__ float gmax[MG_THREADS / 16][16], gsum[MG_THREADS / 16][16];
    {
        const int row = tid & 15, q = tid >> 4;
        constexpr int NG = MG_THREADS / 16;
        float M = -INFINITY;
        for (int r = q; r < nrec; r += NG) M = fmaxf(M, recs[(int64_t)r * DC_REC + row]);
        gmax[q][row] = M;
        __syncthreads();
        M = -INFINITY;
#pragma unroll
        for (int k = 0; k < NG; ++k) M = fmaxf(M, gmax[k][row]);
        float L = 0.f;
        for (int r = q; r < nrec; r += NG) {
            const float m = recs[(int64_t)r * DC_REC + row];
            const float w = m == -INFINITY ? 0.f : fast_exp(m - M);
            wgt[row][r] = w;
            L += w * recs[(int64_t)r * DC_REC + 16 + row];
        }
        gsum[q][row] = L;
        __syncthreads();
        if (tid < 16) {
            float Ls = 0.f;
#pragma unroll
            for (int k = 0; k < NG; ++k) Ls += gsum[k][tid];
            Lr[tid] = Ls;
        }
    }
    __syncthreads();
    // 3. rank-space sum of every row over the coded records, in record order: each thread's
    //    elements (row i / D, coordinate i % D), four records' loads in flight at a time;
    //    rows past `rows` are zero
    {
        float a[EPT];
#pragma unroll
        for (int e = 0; e < EPT; ++e) a[e] = 0.f;
#pragma unroll
        for (int k = 0; k < 4; ++k)
#pragma unroll
            for (int e = 0; e < EPT; ++e) {
                const int row = (tid + e * MG_THREADS) / D;
                if (k < nb0 && row < rows) a[e] += wgt[row][1 + k] * x0[k][e];
            }
        int r = 1 + nb0;
        for (; r + 4 <= nrc; r += 4) {
            float x[4][EPT];
#pragma unroll
            for (int k = 0; k < 4; ++k)
#pragma unroll
                for (int e = 0; e < EPT; ++e) {
                    const int i = tid + e * MG_THREADS;
                    x[k][e] = recs[(int64_t)(r + k) * DC_REC + 32 + i];
                }
#pragma unroll
            for (int k = 0; k < 4; ++k)
#pragma unroll
                for (int e = 0; e < EPT; ++e) {
                    const int row = (tid + e * MG_THREADS) / D;
                    if (row < rows) a[e] += wgt[row][r + k] * x[k][e];
                }
        }
        for (; r < nrc; ++r) {
#pragma unroll
            for (int e = 0; e < EPT; ++e) {
                const int i = tid + e * MG_THREADS, row = i / D;
                if (row < rows) a[e] += wgt[row][r] * recs[(int64_t)r * DC_REC + 32 + i];
            }
        }
#pragma unroll
        for (int e = 0; e < EPT; ++e) {
            const int i = tid + e * MG_THREADS;
            accR[i / D][i % D] = a[e];
        }
    }
    __syncthreads();
    // 4. back-rotation by the slab (wave t: output columns 16 t .. 16 t + 15 of the block), the
    //    original-space records, division by the denominator
    const int wave = tid >> 6, lane = tid & 63;
    if (wave < MG_COLS / 16) {
        const int li = lane & 15, lk = lane >> 4;
        f32x4 o = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
        for (int s = 0; s < D / 4; ++s)
            o = __builtin_amdgcn_mfma_f32_16x16x4f32(accR[li][4 * s + lk], slab[4 * s + lk][16 * wave + li], o, 0, 0, 0);
        const int c = 16 * wave + li;             // C lane: column li, rows 4 lk .. 4 lk + 3
#pragma unroll
        for (int v = 0; v < 4; ++v) {
            const int row = 4 * lk + v;
            if (row >= rows) continue;
            float e = wgt[row][0] * recs[32 + row * D + MG_COLS * cb + c];
            for (int r = nrc; r < nrec; ++r) e += wgt[row][r] * recs[(int64_t)r * DC_REC + 32 + row * D + MG_COLS * cb + c];
            const float val = (o[v] + e) / Lr[row];
            const int qrow = 16 * qt + row;
            const int query = qrow / p.hpg, hh = qrow % p.hpg;
            ET* out = reinterpret_cast<ET*>(p.out) + (int64_t)sq * p.out_seq_stride;
            const int64_t oi = ((int64_t)query * p.H + g * p.hpg + hh) * D + MG_COLS * cb + c;
            if constexpr (F32) out[oi] = val;
            else out[oi] = (uint16_t)f32_to_bf16(val);
        }
    }
}

// ----------------------------------------------------------------------------------------
// Residual codec (Sec. 3.1 Eq. (2)): a coded token's key is its anchors' mean plus the
// truncated projection, so its score is the mean of its 4 anchors' scores plus the rank-space
// product, and its value's anchor part sends a quarter of its softmax weight to each of its
// anchors.  Three more launches around the streaming kernel:
//   anc_qscores  X[unit][a][row] = <q_row, k_a> / sqrt(d) for every anchor (exact rows)
//   anc_xbar     xbar[unit][pos][row] = (1/4) sum of X over the stored position's anchors, the
//                term the streaming kernel adds to each coded score (it also writes the final
//                scores S[unit][pos][row])
//   anc_pieces   per piece of an anchor's list (64 entries): sum of exp(S - F)
//   anc_weights  per anchor: W_a = exp(X_a - F) + (1/4) sum over the positions that use a
//                of exp(S - F) (its pieces)
//   anc_values   one record per (unit, block of anchors) in the original space: for its
//                anchors, acc = sum W_a v_a, l = sum exp(X_a - F), m = F (a bound of every
//                score involved); the merge combines these with the others by log-sum-exp
//                like the exact record.
struct AncDec {
    const varrate_cache* seq;   // unused on the device
    const void* q[DC_SEQ];
    const void* ka[DC_SEQ];
    const void* va[DC_SEQ];
    const uint16_t* snn[DC_SEQ];
    const uint32_t* inv_off[DC_SEQ];
    const uint32_t* inv_pos[DC_SEQ];
    const uint32_t* piece_off[DC_SEQ];
    const uint16_t* piece_anchor[DC_SEQ];
    float* X;          // [unit][na][ns]
    float* XM;         // [unit][ceil(na / 64)][ns] block maxima of X
    float* PW;         // [unit][np_bound][ns] per-piece sums of exp(S - F)
    float* W;          // [unit][na][ns] anchor weights
    float* F;          // [unit][16] the frame
    int64_t np_bound;  // pieces per unit at most: 4 N / 64 + na
    float* xbar;       // [unit][16 total_tiles][ns]
    float* S;          // [unit][16 total_tiles][ns]
    float* part;       // records [unit][nrec][DC_REC]
    int64_t N, na;
    int G, H, hpg, nqt, rows_total, ns, total_tiles, nrec, rec0, ablk, n_ablk;
};

__device__ __forceinline__ void anc_unit(const AncDec& p, int unit, int& sq, int& g, int& qt, int& rows) {
    const int per = p.G * p.nqt;
    sq = unit / per;
    const int gq = unit % per;
    g = gq / p.nqt;
    qt = gq % p.nqt;
    rows = min(16, p.rows_total - 16 * qt);
}

// one thread per (anchor, row): 64 anchors x 4 row groups per workgroup
__global__ __launch_bounds__(256) void anc_qscores(AncDec p) {
    const int blocks = (int)((p.na + 63) / 64);
    const int unit = blockIdx.x / blocks, ab = blockIdx.x % blocks;
    int sq, g, qt, rows;
    anc_unit(p, unit, sq, g, qt, rows);
    const int64_t a = (int64_t)ab * 64 + (threadIdx.x >> 2);
    const int rg = threadIdx.x & 3;
    if (a >= p.na) return;
    const uint16_t* ka = reinterpret_cast<const uint16_t*>(p.ka[sq]) + (a * p.G + g) * D;
    const uint16_t* qb = reinterpret_cast<const uint16_t*>(p.q[sq]);
    float* X = p.X + ((int64_t)unit * p.na + a) * p.ns;
    for (int r = rg; r < p.ns; r += 4) {
        float acc = 0.f;
        if (r < rows) {
            const int qrow = 16 * qt + r;
            const uint16_t* qv = qb + ((int64_t)(qrow / p.hpg) * p.H + g * p.hpg + qrow % p.hpg) * D;
            for (int e = 0; e < D; e += 8) {
                const u32x4 kk = load16(ka + e), qq = load16(qv + e);
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    acc = fmaf(bf_lo(kk[k]), bf_lo(qq[k]), acc);
                    acc = fmaf(bf_hi(kk[k]), bf_hi(qq[k]), acc);
                }
            }
        }
        X[r] = acc * 0.08838834764831845f;   // 1/sqrt(128)
    }
}

// the block maxima of X (per row), for the frame of the anchor weights
__global__ __launch_bounds__(256) void anc_xmax(AncDec p) {
    const int blocks = (int)((p.na + 63) / 64);
    const int unit = blockIdx.x / blocks, ab = blockIdx.x % blocks;
    const int lane = threadIdx.x & 63, r = threadIdx.x >> 6;   // 4 waves: rows r, r + 4, ...
    const int64_t a = (int64_t)ab * 64 + lane;
    const float* X = p.X + (int64_t)unit * p.na * p.ns;
    for (int rr = r; rr < p.ns; rr += 4) {
        float m = a < p.na ? X[a * p.ns + rr] : -INFINITY;
#pragma unroll
        for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
        if (lane == 0) p.XM[((int64_t)unit * blocks + ab) * p.ns + rr] = m;
    }
}

// one thread per (stored position, row group)
__global__ __launch_bounds__(256) void anc_xbar(AncDec p) {
    const int npos = 16 * p.total_tiles;
    const int blocks = (npos + 63) / 64;
    const int unit = blockIdx.x / blocks, pb = blockIdx.x % blocks;
    int sq, g, qt, rows;
    anc_unit(p, unit, sq, g, qt, rows);
    const int64_t pos = (int64_t)pb * 64 + (threadIdx.x >> 2);
    const int rg = threadIdx.x & 3;
    if (pos >= npos) return;
    float* xb = p.xbar + ((int64_t)unit * npos + pos) * p.ns;
    const float* X = p.X + (int64_t)unit * p.na * p.ns;
    if (pos >= p.N) {
        for (int r = rg; r < p.ns; r += 4) xb[r] = 0.f;
        return;
    }
    const uint16_t* nn = p.snn[sq] + pos * 4;
    const int64_t a0 = nn[0], a1 = nn[1], a2 = nn[2], a3 = nn[3];
    for (int r = rg; r < p.ns; r += 4)
        xb[r] = (((X[a0 * p.ns + r] + X[a1 * p.ns + r]) + X[a2 * p.ns + r]) + X[a3 * p.ns + r]) * 0.25f;
}

// The frame F[row] of the anchor weights: an upper bound of every score they involve, the
// largest of the anchors' own scores and of the streaming records' running maxima + 8 (each
// coded score exceeds its workgroup's running maximum by at most 8).  All 256 threads scan
// (thread -> row tid % 16, every 16th record and block maximum), then a max over the 16
// partial maxima; a maximum does not depend on the order, so every workgroup that computes
// it gets the same F.
__device__ __forceinline__ void anc_frame(const AncDec& p, int unit, int rows, float* F_s) {
    __shared__ float part_m[16][17], part_x[16][17];
    const int tid = threadIdx.x, r = tid & 15, k = tid >> 4;
    const float* recs = p.part + (int64_t)unit * p.nrec * DC_REC;
    const int xb = (int)((p.na + 63) / 64);
    const float* XM = p.XM + (int64_t)unit * xb * p.ns;
    float m = -INFINITY, mx = -INFINITY;
    if (r < rows) {
        for (int x = k; x < p.rec0; x += 16) m = fmaxf(m, recs[(int64_t)x * DC_REC + r]);
        for (int b = k; b < xb; b += 16) mx = fmaxf(mx, XM[b * p.ns + r]);
    }
    part_m[k][r] = m;
    part_x[k][r] = mx;
    __syncthreads();
    if (tid < 16) {
        m = -INFINITY;
        mx = -INFINITY;
        for (int j = 0; j < 16; ++j) {
            m = fmaxf(m, part_m[j][tid]);
            mx = fmaxf(mx, part_x[j][tid]);
        }
        F_s[tid] = tid < rows ? fmaxf(m + 8.f, mx) : 0.f;
    }
    __syncthreads();
}

// Four threads per list piece (at most 64 entries, 16 each, all loads in flight), then a
// fixed two-step butterfly: PW[P][row] = sum over the piece of exp(S - F).  The first
// workgroup of each unit also stores F for the kernels after it.
constexpr int AP_T = 256;
constexpr int AP_PIECES = AP_T / 4;   // pieces per workgroup
__global__ __launch_bounds__(AP_T) void anc_pieces(AncDec p) {
    __shared__ float F_s[16];
    const int blocks = (int)((p.np_bound + AP_PIECES - 1) / AP_PIECES);
    const int unit = blockIdx.x / blocks, pb = blockIdx.x % blocks;
    int sq, g, qt, rows;
    anc_unit(p, unit, sq, g, qt, rows);
    anc_frame(p, unit, rows, F_s);
    if (pb == 0 && threadIdx.x < 16) p.F[unit * 16 + threadIdx.x] = F_s[threadIdx.x];
    const int64_t P = (int64_t)pb * AP_PIECES + (threadIdx.x >> 2);
    const int sub = threadIdx.x & 3;
    const uint32_t npieces = p.piece_off[sq][p.na];
    // whole quads leave together, so the butterfly below sees all four lanes
    if (P >= (int64_t)npieces) return;
    const int ns = p.ns;
    const uint32_t a = p.piece_anchor[sq][P];
    const uint32_t j = (uint32_t)P - p.piece_off[sq][a];
    const uint32_t e_end = p.inv_off[sq][a + 1];
    const uint32_t e0 = min(p.inv_off[sq][a] + 64 * j + 16 * sub, e_end);
    const uint32_t e1 = min(e0 + 16, e_end);
    const uint32_t* inv = p.inv_pos[sq];
    const float* S = p.S + (int64_t)unit * 16 * p.total_tiles * ns;
    float F[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) F[r] = F_s[r];
    uint32_t pos[16];
#pragma unroll
    for (int u = 0; u < 16; ++u) pos[u] = e0 + u < e1 ? inv[e0 + u] : 0u;
    float sh[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) sh[r] = 0.f;
#pragma unroll
    for (int u = 0; u < 16; ++u) {
        const bool ok = e0 + u < e1;
        const f32x4* sp = reinterpret_cast<const f32x4*>(S + (int64_t)pos[u] * ns);
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
            if (4 * r4 < ns && ok) {
                const f32x4 v = sp[r4];
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    if (4 * r4 + k < rows) sh[4 * r4 + k] += fast_exp(v[k] - F[4 * r4 + k]);
            }
        }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        if (r < ns) {
            sh[r] += __shfl_xor(sh[r], 1, 64);
            sh[r] += __shfl_xor(sh[r], 2, 64);
        }
    }
    if (sub == 0) {
        float* pw = p.PW + ((int64_t)unit * p.np_bound + P) * ns;
#pragma unroll
        for (int r = 0; r < 16; ++r)
            if (r < ns) pw[r] = sh[r];
    }
}

// A wave per anchor: W_a = exp(X_a - F) + (1/4) sum of its pieces' PW (lanes take every 64th
// piece, then a fixed butterfly).  Writes W[unit][a][row] and the anchor's own mass
// exp(X_a - F) over X (read only here, by the same lane).
constexpr int AW_T = 256;
__global__ __launch_bounds__(AW_T) void anc_weights(AncDec p) {
    const int blocks = (int)((p.na + AW_T / 64 - 1) / (AW_T / 64));
    const int unit = blockIdx.x / blocks, ab = blockIdx.x % blocks;
    int sq, g, qt, rows;
    anc_unit(p, unit, sq, g, qt, rows);
    const int lane = threadIdx.x & 63;
    const int64_t a = (int64_t)ab * (AW_T / 64) + (threadIdx.x >> 6);
    if (a >= p.na) return;   // whole waves
    const int ns = p.ns;
    const uint32_t P0 = p.piece_off[sq][a], P1 = p.piece_off[sq][a + 1];
    const float* PW = p.PW + (int64_t)unit * p.np_bound * ns;
    float sh[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) sh[r] = 0.f;
    for (uint32_t P = P0 + lane; P < P1; P += 64) {
        const f32x4* pw = reinterpret_cast<const f32x4*>(PW + (int64_t)P * ns);
#pragma unroll
        for (int r4 = 0; r4 < 4; ++r4) {
            if (4 * r4 < ns) {
                const f32x4 v = pw[r4];
#pragma unroll
                for (int k = 0; k < 4; ++k) sh[4 * r4 + k] += v[k];
            }
        }
    }
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        if (r < rows) {
            float v = sh[r];
#pragma unroll
            for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
            sh[r] = v;
        }
    }
    if (lane < ns) {
        const int r = lane;
        float shr = 0.f;
#pragma unroll
        for (int rr = 0; rr < 16; ++rr) shr = rr == r ? sh[rr] : shr;
        float* X = p.X + ((int64_t)unit * p.na + a) * ns;
        const float own = r < rows ? fast_exp(X[r] - p.F[unit * 16 + r]) : 0.f;
        X[r] = own;
        p.W[((int64_t)unit * p.na + a) * ns + r] = r < rows ? own + 0.25f * shr : 0.f;
    }
}

// A workgroup per (unit, block of AV_A anchors): the value sums over the block's anchors
// (value rows and weights staged in LDS) and its record.
constexpr int AV_T = 256;
constexpr int AV_A = 64;                          // anchors per workgroup
__global__ __launch_bounds__(AV_T) void anc_values(AncDec p) {
    __shared__ float red[16];
    __shared__ float W[AV_A][17];
    __shared__ float own_s[AV_A][17];
    __shared__ __attribute__((aligned(16))) uint16_t vrow[AV_A][D];
    const int unit = blockIdx.x / p.n_ablk, ab = blockIdx.x % p.n_ablk;
    int sq, g, qt, rows;
    anc_unit(p, unit, sq, g, qt, rows);
    const int tid = threadIdx.x;
    const int64_t a_lo = (int64_t)ab * AV_A;
    const int nact = (int)min<int64_t>(AV_A, p.na - a_lo);
    const int ns = p.ns;
    // the block's value rows, weights and own masses into LDS (all loads in flight together)
    {
        const uint16_t* va = reinterpret_cast<const uint16_t*>(p.va[sq]);
        for (int k = tid; k < nact * (D / 8); k += AV_T) {
            const int j = k / (D / 8), e = 8 * (k % (D / 8));
            *reinterpret_cast<u32x4*>(&vrow[j][e]) = load16(va + ((a_lo + j) * p.G + g) * D + e);
        }
        const float* Wg = p.W + ((int64_t)unit * p.na + a_lo) * ns;
        const float* Og = p.X + ((int64_t)unit * p.na + a_lo) * ns;
        for (int k = tid; k < AV_A * 16; k += AV_T) {
            const int j = k >> 4, r = k & 15;
            const bool ok = j < nact && r < ns;
            W[j][r] = ok ? Wg[j * ns + r] : 0.f;
            own_s[j][r] = ok ? Og[j * ns + r] : 0.f;
        }
    }
    __syncthreads();
    // the anchors' own softmax mass, in anchor order
    if (tid < 16) {
        float l = 0.f;
        for (int j = 0; j < nact; ++j) l += own_s[j][tid];
        red[tid] = l;
    }
    // ---- the value sums: thread -> column c, rows rh, rh + 2, ... (anchors in order)
    const int c = tid & (D - 1), rh = tid >> 7;
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < nact; ++j) {
        const float v = bf16_to_f32(vrow[j][c]);
#pragma unroll
        for (int k = 0; k < 8; ++k) acc[k] = fmaf(W[j][rh + 2 * k], v, acc[k]);
    }
    __syncthreads();
    // ---- the record: m = F, l = the anchors' own mass, acc in the original space
    float* rec = p.part + ((int64_t)unit * p.nrec + p.rec0 + ab) * DC_REC;
    if (tid < 16) {
        rec[tid] = tid < rows ? p.F[unit * 16 + tid] : -INFINITY;
        rec[16 + tid] = tid < rows ? red[tid] : 0.f;
    }
#pragma unroll
    for (int k = 0; k < 8; ++k) {
        const int r = rh + 2 * k;
        if (r < ((rows + 3) & ~3)) rec[32 + r * D + c] = r < rows ? acc[k] : 0.f;
    }
}

// ----------------------------------------------------------------------------------------
struct DecPlan {
    int nqt, n_chunks, cpw, n_wg, tpw, total_tiles;
    int nrec, n_ablk, ns;      // records per unit; residual codec: anchor records, score rows
    int64_t na;
    bool ring;                 // decode_ring_kernel (n_wg = its workgroups per unit)
    int rt;                    // ring kernel: row tiles per wave (2 for a batch of query rows)
};

// allow_ring: bf16 coefficients of the plain codec go to the ring kernel when every wave's
// tile run fits its offset registers
static DecPlan plan_decode(const varrate_shape& sh, int S, int Q, bool allow_ring = true) {
    DecPlan pl;
    const int64_t N = coded_count(sh);
    const int rows_total = Q * (sh.H / sh.G);
    pl.nqt = (rows_total + 15) / 16;
    pl.n_chunks = (int)((N + CHUNK - 1) / CHUNK);
    const int64_t last = N - (int64_t)(pl.n_chunks - 1) * CHUNK;
    pl.total_tiles = 16 * (pl.n_chunks - 1) + (int)((last + 15) / 16);
    const int units = (S < DC_SEQ ? S : DC_SEQ) * sh.G * pl.nqt;
    // coded workgroups + one exact workgroup per unit: about two workgroups per CU, at
    // least one tile per wave, at most (DC_MAX_CPW - 1) chunks of tiles per workgroup
    int n_wg = 512 / (units > 0 ? units : 1) - 1;
    const int by_waves = (pl.total_tiles + DC_WAVES - 1) / DC_WAVES;
    const int max_tpw = (DC_MAX_CPW - 1) * 16;
    const int by_span = (pl.total_tiles + max_tpw - 1) / max_tpw;
    n_wg = n_wg > by_waves ? by_waves : n_wg;
    n_wg = n_wg < by_span ? by_span : n_wg;
    n_wg = n_wg < 1 ? 1 : n_wg;
    pl.tpw = (pl.total_tiles + n_wg - 1) / n_wg;
    pl.n_wg = (pl.total_tiles + pl.tpw - 1) / pl.tpw;
    pl.cpw = (pl.tpw + 15) / 16 + 1;    // chunks a tile range can touch
    pl.na = anchor_count(sh);
    pl.n_ablk = (int)((pl.na + AV_A - 1) / AV_A);
    pl.nrec = pl.n_wg + 1 + pl.n_ablk;
    pl.ns = rows_total < 16 ? (rows_total + 3) & ~3 : 16;
    pl.ring = false;
    pl.rt = pl.nqt >= 2 ? 2 : 1;
    if (allow_ring && sh.dtype == VARRATE_BF16 && !sh.rope && pl.na == 0 && units > 0) {
        // the ring kernel's units: (sequence, KV head, group of rt row tiles)
        const int ru = units / pl.nqt * ((pl.nqt + pl.rt - 1) / pl.rt);
        const int wpu = DR_CUS / ru > 1 ? DR_CUS / ru : 1;
        const int ncw_min = wpu == 1 ? DR_WAVES - 4 : DR_WAVES * wpu - DR_WAVES;   // n_xw at its cap
        if ((pl.total_tiles + ncw_min - 1) / ncw_min <= DR_MAX_TPW) {
            pl.ring = true;
            pl.n_wg = wpu;
            pl.nrec = wpu + 1;
        }
    }
    return pl;
}

// Workspace: the partial records of every (sequence, KV head, row tile).
size_t decode_units(const varrate_shape& sh, int S, int Q) {
    return (size_t)S * sh.G * plan_decode(sh, S, Q).nqt;
}

bool decode_supported(const varrate_shape& sh, int S, int Q) {
    return plan_decode(sh, S, Q, false).nrec <= DC_MAX_REC && plan_decode(sh, S, Q).nrec <= DC_MAX_REC;
}

// Residual codec buffers after the records: X [units][na][ns], xbar and S [units][16 tiles][ns],
// XM [units][na / 64][ns], PW [units][pieces][ns], W [units][na][ns], F [units][16]
static inline int64_t anc_np_bound(const DecPlan& pl, int64_t N) { return 4 * N / 64 + pl.na; }
static size_t anc_dec_bytes(const DecPlan& pl, size_t units, int64_t N) {
    if (!pl.na) return 0;
    return 2 * align256(units * pl.na * pl.ns * 4) + 2 * align256(units * 16 * (size_t)pl.total_tiles * pl.ns * 4) +
           align256(units * ((pl.na + 63) / 64) * pl.ns * 4) + align256(units * anc_np_bound(pl, N) * pl.ns * 4) +
           align256(units * 16 * 4);
}

size_t decode_ws_bytes(const varrate_shape& sh, int S, int Q) {
    DecPlan pl = plan_decode(sh, S, Q, false);
    const DecPlan pr = plan_decode(sh, S, Q);
    if (pr.nrec > pl.nrec) pl.nrec = pr.nrec;     // room for either kernel's records
    const size_t units = (size_t)S * sh.G * pl.nqt;
    const size_t rope = sh.rope ? align256((size_t)sh.G * ROPE_FRAG_BYTES) + align256(D * sizeof(float)) : 0;
    return align256(units * pl.nrec * DC_REC * sizeof(float)) + anc_dec_bytes(pl, units, coded_count(sh)) + rope;
}

hipError_t launch_decode(const varrate_shape& sh, const varrate_cache* caches, int S, const void* q,
                         int Q, const float* PK, const float* PV, void* out, uint8_t* ws,
                         hipStream_t st, bool reuse_group_region, const varrate_qcache* qcaches) {
    const int qb = qcaches ? qcaches[0].bits : 0;
    DecPlan pl = plan_decode(sh, S, Q, qb == 0);
    if (qb != 0 && qb != 3 && qb != 4 && qb != 8) return hipErrorInvalidValue;
    if (qb != 0 && sh.dtype != VARRATE_BF16) return hipErrorInvalidValue;
    const bool anc = pl.na > 0;
    typedef void (*DecFn)(DecParams);
    DecFn kfn;
    const bool rope = sh.rope != 0;
    if (rope && (qb != 0 || anc)) return hipErrorInvalidValue;
    if (rope) kfn = sh.dtype != VARRATE_BF16 ? decode_kernel<true, 0, false, true> : decode_kernel<false, 0, false, true>;
    else if (sh.dtype != VARRATE_BF16) kfn = decode_kernel<true, 0, false>;
    else if (!anc) kfn = qb == 3 ? decode_kernel<false, 3, false> : qb == 4 ? decode_kernel<false, 4, false>
                       : qb == 8 ? decode_kernel<false, 8, false> : decode_kernel<false, 0, false>;
    else kfn = qb == 3 ? decode_kernel<false, 3, true> : qb == 4 ? decode_kernel<false, 4, true>
             : qb == 8 ? decode_kernel<false, 8, true> : decode_kernel<false, 0, true>;
    const int hpg = sh.H / sh.G;
    const int rows_total = Q * hpg;
    const size_t units_all = (size_t)S * sh.G * pl.nqt;
    if (pl.nrec > DC_MAX_REC) return hipErrorInvalidValue;
    float* part = (float*)ws;
    // residual codec: X, xbar and S after the records
    float *Xb = nullptr, *xbarb = nullptr, *Sb = nullptr, *XMb = nullptr, *PWb = nullptr, *Wb = nullptr,
          *Fb = nullptr;
    const int64_t np_bound = anc_np_bound(pl, coded_count(sh));
    if (anc) {
        if (reuse_group_region) return hipErrorInvalidValue;   // no fixed scratch for it
        uint8_t* b = ws + align256(units_all * pl.nrec * DC_REC * sizeof(float));
        Xb = (float*)b;
        b += align256(units_all * pl.na * pl.ns * 4);
        xbarb = (float*)b;
        b += align256(units_all * 16 * (size_t)pl.total_tiles * pl.ns * 4);
        Sb = (float*)b;
        b += align256(units_all * 16 * (size_t)pl.total_tiles * pl.ns * 4);
        XMb = (float*)b;
        b += align256(units_all * ((pl.na + 63) / 64) * pl.ns * 4);
        PWb = (float*)b;
        b += align256(units_all * np_bound * pl.ns * 4);
        Wb = (float*)b;
        b += align256(units_all * pl.na * pl.ns * 4);
        Fb = (float*)b;
    }
    // rotary keys: the basis fragments and the frequency table after the records, prepared
    // once per call
    const u32x4* rfrag = nullptr;
    const float* rfreq = nullptr;
    hipError_t e;
    if (rope) {
        if (reuse_group_region) return hipErrorInvalidValue;   // no fixed scratch for it
        uint8_t* b = ws + align256(units_all * pl.nrec * DC_REC * sizeof(float));
        rfrag = reinterpret_cast<const u32x4*>(b);
        float* fq = reinterpret_cast<float*>(b + align256((size_t)sh.G * ROPE_FRAG_BYTES));
        rfreq = fq;
        e = launch_rope_prep(sh, PK, b, fq, st);
        if (e != hipSuccess) return e;
    }
    const size_t es = sh.dtype == VARRATE_BF16 ? 2 : 4;
    const size_t qstride = (size_t)Q * sh.H * D * es;
    const size_t lds = pl.ring ? (pl.rt == 2 ? dr_smem<2>() : dr_smem<1>()) : decode_smem_bytes(pl.cpw, rope);
    if (pl.ring) kfn = pl.rt == 2 ? decode_ring_kernel<2> : decode_ring_kernel<1>;
    e = ensure_lds_limit((const void*)kfn, lds);
    if (e != hipSuccess) return e;
    for (int s0 = 0; s0 < S; s0 += DC_SEQ) {
        const int ns = S - s0 < DC_SEQ ? S - s0 : DC_SEQ;
        DecParams prm;
        for (int i = 0; i < ns; ++i) {
            const varrate_cache& c = caches[s0 + i];
            // quantised: the code streams and their (byte) chunk bases replace the coefficients
            const void* ck = qb ? qcaches[s0 + i].code_k : c.coef_k;
            const void* cv = qb ? qcaches[s0 + i].code_v : c.coef_v;
            const uint32_t* co = qb ? qcaches[s0 + i].qchunk_off : c.chunk_off;
            prm.seq[i] = DecSeq{ck, cv, c.srank, co, c.k_exact, c.v_exact,
                                (const uint8_t*)q + (s0 + i) * qstride, (uint8_t*)out + (s0 + i) * qstride,
                                c.n_exact, c.sidx};
        }
        for (int i = ns; i < DC_SEQ; ++i) prm.seq[i] = prm.seq[0];
        prm.PK = PK;
        prm.rfrag = rfrag;
        prm.rfreq = rfreq;
        prm.PV = PV;
        // launch groups run in stream order, so with reuse_group_region every group's records
        // go to the start of the buffer (the previous group's merge has finished reading them)
        prm.part = reuse_group_region ? part : part + (size_t)s0 * sh.G * pl.nqt * pl.nrec * DC_REC;
        prm.N = coded_count(sh);
        prm.coef_stride = qb ? qcaches[s0].q_stride / 2 : caches[s0].coef_stride;   // 2-byte units
        prm.cap = caches[s0].cap;
        prm.G = sh.G;
        prm.H = sh.H;
        prm.hpg = hpg;
        prm.nqt = pl.nqt;
        prm.rows_total = rows_total;
        prm.n_chunks = pl.n_chunks;
        prm.cpw = pl.cpw;
        prm.n_wg = pl.n_wg;
        prm.tpw = pl.tpw;
        prm.total_tiles = pl.total_tiles;
        prm.units = ns * sh.G * pl.nqt;
        prm.nrec = pl.nrec;
        prm.ns = pl.ns;
        prm.xbar = nullptr;
        prm.S = nullptr;
        AncDec ad;
        if (pl.na) {
            const size_t u0 = (size_t)s0 * sh.G * pl.nqt;
            prm.xbar = xbarb + u0 * 16 * pl.total_tiles * pl.ns;
            prm.S = Sb + u0 * 16 * pl.total_tiles * pl.ns;
            ad.seq = nullptr;
            for (int i = 0; i < DC_SEQ; ++i) {
                const int si = s0 + (i < ns ? i : 0);
                const varrate_cache& c = caches[si];
                ad.q[i] = (const uint8_t*)q + si * qstride;
                ad.ka[i] = c.k_anchor;
                ad.va[i] = c.v_anchor;
                ad.snn[i] = c.snn;
                ad.inv_off[i] = c.inv_off;
                ad.inv_pos[i] = c.inv_pos;
                ad.piece_off[i] = c.piece_off;
                ad.piece_anchor[i] = c.piece_anchor;
            }
            ad.X = Xb + u0 * pl.na * pl.ns;
            ad.XM = XMb + u0 * ((pl.na + 63) / 64) * pl.ns;
            ad.PW = PWb + u0 * np_bound * pl.ns;
            ad.W = Wb + u0 * pl.na * pl.ns;
            ad.F = Fb + u0 * 16;
            ad.np_bound = np_bound;
            ad.xbar = const_cast<float*>(prm.xbar);
            ad.S = prm.S;
            ad.part = prm.part;
            ad.N = prm.N;
            ad.na = pl.na;
            ad.G = sh.G;
            ad.H = sh.H;
            ad.hpg = hpg;
            ad.nqt = pl.nqt;
            ad.rows_total = rows_total;
            ad.ns = pl.ns;
            ad.total_tiles = pl.total_tiles;
            ad.nrec = pl.nrec;
            ad.rec0 = pl.n_wg + 1;
            ad.ablk = AV_A;
            ad.n_ablk = pl.n_ablk;
            anc_qscores<<<(unsigned)(prm.units * ((pl.na + 63) / 64)), 256, 0, st>>>(ad);
            anc_xmax<<<(unsigned)(prm.units * ((pl.na + 63) / 64)), 256, 0, st>>>(ad);
            anc_xbar<<<(unsigned)(prm.units * ((16 * pl.total_tiles + 63) / 64)), 256, 0, st>>>(ad);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        prm.wpu = pl.n_wg;
        prm.n_xw = 0;
        if (pl.ring) {
            // exact waves in proportion to the exact rows' share of the streamed bytes (the coded
            // share estimated from the budget and the tiles' measured 6% padding), at least one,
            // at most one per exact tile and half the unit's waves when it has one workgroup
            int64_t nx = 0;
            for (int i = 0; i < ns; ++i) nx = caches[s0 + i].n_exact > nx ? caches[s0 + i].n_exact : nx;
            const int X = (int)((nx + 15) / 16);
            const double xb = (double)nx * D, cb = (double)caches[s0].B * 1.06;
            int nxw = (int)(DR_WAVES * pl.n_wg * xb / (xb + cb) + 0.5);
            const int cap_x = pl.n_wg == 1 ? DR_WAVES / 2 : DR_WAVES;
            nxw = nxw > cap_x ? cap_x : nxw;
            nxw = nxw > X ? X : nxw;
            prm.n_xw = nxw < 1 ? 1 : nxw;
        }
        const unsigned nblk = pl.ring ? (unsigned)(prm.units / pl.nqt * ((pl.nqt + pl.rt - 1) / pl.rt) * pl.n_wg)
                                      : (unsigned)(prm.units * (pl.n_wg + 1));
        kfn<<<nblk, pl.ring ? DR_THREADS : DC_THREADS, lds, st>>>(prm);
        e = hipGetLastError();
        if (e != hipSuccess) return e;
        if (pl.na) {
            anc_pieces<<<(unsigned)(prm.units * ((np_bound + AP_PIECES - 1) / AP_PIECES)), AP_T, 0, st>>>(ad);
            anc_weights<<<(unsigned)(prm.units * ((pl.na + AW_T / 64 - 1) / (AW_T / 64))), AW_T, 0, st>>>(ad);
            anc_values<<<(unsigned)(prm.units * pl.n_ablk), AV_T, 0, st>>>(ad);
            e = hipGetLastError();
            if (e != hipSuccess) return e;
        }
        MergeParams mp;
        mp.part = prm.part;
        mp.PV = PV;
        mp.out = (uint8_t*)out + s0 * qstride;
        mp.out_seq_stride = (int64_t)Q * sh.H * D;
        mp.G = sh.G;
        mp.H = sh.H;
        mp.hpg = hpg;
        mp.nqt = pl.nqt;
        mp.rows_total = rows_total;
        mp.n_wg = pl.n_wg;
        mp.rpu = rows_total < 16 ? rows_total : 16;
        mp.nrec = pl.nrec;
        // units of more than 8 query rows (batches of queries): one workgroup per (unit, column
        // block) for all rows; up to 8 rows the per-row spread keeps more workgroups busy
        // (Qwen's 7 rows per KV head: 0.80 against 1.07 ms per 28-layer step)
        const bool by_rows = mp.rpu > 8;
        const unsigned nmerge = (unsigned)(ns * sh.G * pl.nqt * (by_rows ? 1 : mp.rpu) * MG_CB);
        {
            // XCD-aware order when the heads spread evenly over the 8 XCDs
            const int per_head = ns * pl.nqt * (by_rows ? 1 : mp.rpu) * MG_CB;
            const int m = sh.G < 8 ? 8 / sh.G : 1;
            const bool even = (sh.G % 8 == 0) || (8 % sh.G == 0 && per_head % m == 0);
            mp.xcd_m = even && nmerge % 8 == 0 ? m : 0;
        }
        if (by_rows) {
            if (sh.dtype == VARRATE_BF16) decode_merge_rows_kernel<false><<<nmerge, MG_THREADS, 0, st>>>(mp);
            else decode_merge_rows_kernel<true><<<nmerge, MG_THREADS, 0, st>>>(mp);
        } else if (sh.dtype == VARRATE_BF16) {
            decode_merge_kernel<false><<<nmerge, MG_THREADS, 0, st>>>(mp);
        } else {
            decode_merge_kernel<true><<<nmerge, MG_THREADS, 0, st>>>(mp);
        }
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    return hipSuccess;
}


// ----------------------------------------------------------------------------------------
// Decode without a caller workspace: the partial records live in a fixed device array.
// Each device holds its own copy of `scratch` at its own address, looked up once per device
// with hipGetSymbolAddress; host code only ever passes that address (the array's name is a
// host-side stand-in).  The launch groups of one call reuse the array in stream order.  The
// records need no clearing: every record the merge reads is written by the streaming launch
// of the same group first.
static __device__ __attribute__((aligned(256))) uint8_t scratch[VARRATE_DECODE_SCRATCH_BYTES];

constexpr int SCRATCH_MAX_DEVICES = 64;
static std::mutex scratch_mu;
static void* scratch_addr[SCRATCH_MAX_DEVICES];

size_t decode_group_bytes(const varrate_shape& sh, int S, int Q) {
    const DecPlan pl = plan_decode(sh, S, Q, false), pr = plan_decode(sh, S, Q);
    const int ns = S < DC_SEQ ? S : DC_SEQ;
    const int nrec = pr.n_wg + 1 > pl.n_wg + 1 ? pr.n_wg + 1 : pl.n_wg + 1;
    return (size_t)ns * sh.G * pl.nqt * nrec * DC_REC * sizeof(float);
}

hipError_t decode_scratch(uint8_t** out) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= SCRATCH_MAX_DEVICES) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(scratch_mu);
    if (!scratch_addr[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        scratch_addr[dev] = p;
    }
    *out = (uint8_t*)scratch_addr[dev];
    return hipSuccess;
}

}  // namespace vr
