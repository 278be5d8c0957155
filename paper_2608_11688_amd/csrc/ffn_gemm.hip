// Expert FFN for two or more tokens (apex_moe_ffn, batch >= 2): a grouped GEMM on the
// matrix cores.
//
// up_gemm and down_gemm take tokens as the M dimension (tiles of 16, padded), weight
// rows as N and the hidden / intermediate dimension as K, with v_mfma_f32_16x16x32_bf16
// (activations rounded to bf16, fp32 accumulation).  A workgroup owns 64 weight rows of
// one expert (blockIdx.y is the expert id; experts without a slot exit at once) and
// finds that expert's (token, position) pairs itself from exec_idx, in pair order, while
// its first weight block loads (an expert without tokens then exits and drops that
// block).  When a projection has too few row tiles to keep the chip's loads in flight
// (plan_for), its K range is split over blockIdx.z and each split writes fp32 partial
// sums:
//   * up_gemm with one split writes h = bf16(silu(W1 x) * (W3 x)) per pair; with several
//     it writes the partial W1 x and W3 x, and swiglu_reduce adds them (in split order)
//     into the same bf16 h, once, before down_gemm reads it from every row tile;
//   * down_gemm writes per-split, per-pair outputs; combine_pairs adds the splits and the
//     gated positions of each token in a fixed order.
// Slots hold bf16 weights (apex_pack_expert), E4M3 codes with fp32 row scales
// (apex_pack_expert_fp8) or MXFP4 codes with a power-of-two scale per block of 32
// (apex_pack_expert_mxfp4).  E4M3 and MXFP4 codes are staged in LDS as bytes and widened
// to bf16 exactly at fragment read (MXFP4 with its block scales applied); the E4M3 row
// scales multiply the outputs.  Every executed expert's weights are read once per call
// whatever the number of tokens routed to it, and no atomics are used, so results are
// deterministic.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "ffn_device.h"
#include "ffn_internal.h"

namespace {

using apex::ffn::kWave;
using apex::ffn::ld_stream;
using apex::ffn::silu;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;
constexpr int kRows = 64;          // weight rows per workgroup tile
constexpr int kKB = 128;           // K per staged block
constexpr int kLdsRow = kKB + 8;   // +16 B per row: the 16 rows of a fragment read hit distinct banks
constexpr int kMaxSplit = 4;

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

__device__ __forceinline__ uint4 pack_bf16(float a0, float a1, float a2, float a3, float a4,
                                           float a5, float a6, float a7) {
    bf16x8 v;
    v[0] = (__bf16)a0; v[1] = (__bf16)a1; v[2] = (__bf16)a2; v[3] = (__bf16)a3;
    v[4] = (__bf16)a4; v[5] = (__bf16)a5; v[6] = (__bf16)a6; v[7] = (__bf16)a7;
    return __builtin_bit_cast(uint4, v);
}

// Component-wise select: a select of the whole vector struct is lowered through
// private memory by the compiler.
__device__ __forceinline__ uint4 keep_if(uint4 v, bool c) {
    return make_uint4(c ? v.x : 0u, c ? v.y : 0u, c ? v.z : 0u, c ? v.w : 0u);
}

// Activation sources: 8 consecutive K values of one row.  load() fetches them as they are
// stored and to_bf16() converts them when the block is staged in LDS, so that no
// arithmetic follows a load directly (which would make the compiler wait for it, and for
// every older load, before the matrix cores work on the previous block).
struct ActF32 {          // fp32 rows (the FFN input x), rounded to bf16 at staging
    struct Raw {
        float4 a, b;
    };
    static __device__ __forceinline__ Raw load(const void *row, int kc) {
        const float4 *p = reinterpret_cast<const float4 *>(static_cast<const float *>(row) + kc);
        return Raw{p[0], p[1]};
    }
    static __device__ __forceinline__ uint4 to_bf16(const Raw &r) {
        return pack_bf16(r.a.x, r.a.y, r.a.z, r.a.w, r.b.x, r.b.y, r.b.z, r.b.w);
    }
};
struct ActBf16 {         // bf16 rows (h)
    using Raw = uint4;
    static __device__ __forceinline__ Raw load(const void *row, int kc) {
        return *reinterpret_cast<const uint4 *>(static_cast<const uint16_t *>(row) + kc);
    }
    static __device__ __forceinline__ uint4 to_bf16(const Raw &r) { return r; }
};
// h = bf16(silu(u) * v) of 8 consecutive values from SU split partials: u of split s at
// r + 2s*stride, v at r + (2s+1)*stride, the splits added in order.
template <int SU>
__device__ __forceinline__ uint4 swiglu8(const float *r, size_t stride) {
    float u[8], v[8];
#pragma unroll
    for (int c = 0; c < 8; ++c) u[c] = v[c] = 0.f;
#pragma unroll
    for (int s = 0; s < SU; ++s) {
        const float4 *pu = reinterpret_cast<const float4 *>(r + 2 * s * stride);
        const float4 *pv = reinterpret_cast<const float4 *>(r + (2 * s + 1) * stride);
        const float4 u0 = pu[0], u1 = pu[1], v0 = pv[0], v1 = pv[1];
        u[0] += u0.x; u[1] += u0.y; u[2] += u0.z; u[3] += u0.w;
        u[4] += u1.x; u[5] += u1.y; u[6] += u1.z; u[7] += u1.w;
        v[0] += v0.x; v[1] += v0.y; v[2] += v0.z; v[3] += v0.w;
        v[4] += v1.x; v[5] += v1.y; v[6] += v1.z; v[7] += v1.w;
    }
    return pack_bf16(silu(u[0]) * v[0], silu(u[1]) * v[1], silu(u[2]) * v[2],
                     silu(u[3]) * v[3], silu(u[4]) * v[4], silu(u[5]) * v[5],
                     silu(u[6]) * v[6], silu(u[7]) * v[7]);
}

// Weight formats of a slot.
// kUpGroups: workgroups the gate/up projection's K splits aim at (see plan_for);
// kKPerElem: K values per element of T; kFp8: fp32 row scales after the codes;
// kBlockScale: one scale byte per 32 K values of a row;
// kCodes: the codes go to LDS as bytes, in K blocks of kb<MT>() values, and are widened
// at fragment read; otherwise bf16 tiles of kKB,
// where one 16-byte load covers 8 K values of a row, kThrPerRow threads cover a block of
// the row and kRowsPerPass rows are loaded per pass of the workgroup.
struct WBf16 {           // apex_pack_expert slots: bf16 weights
    using T = uint16_t;
    [[maybe_unused]] static constexpr bool kFp8 = false, kBlockScale = false, kCodes = false;
    template <int MT> static constexpr int kb() { return kKB; }
    static constexpr int kUpGroups = 400;
    static constexpr int kKPerElem = 1;
    static constexpr int kThrPerRow = kKB / 8, kRowsPerPass = kThreads / kThrPerRow;
    static constexpr int kLoads = kRows / kRowsPerPass;
};
struct WE4M3 {           // apex_pack_expert_fp8 slots: E4M3 codes, fp32 row scales after them
    using T = uint8_t;
    static constexpr bool kFp8 = true, kBlockScale = false, kCodes = true;
    // 256 bytes per row with one token tile, 128 with more (a smaller activation tile)
    template <int MT> static constexpr int kb() { return MT == 1 ? 256 : 128; }
    static constexpr int kUpGroups = 800;
    static constexpr int kKPerElem = 1;
};
struct WMxfp4 {          // apex_pack_expert_mxfp4 slots: two E2M1 codes per byte, block scales
    using T = uint8_t;
    static constexpr bool kFp8 = false, kBlockScale = true, kCodes = true;
    // 256 bytes per row with one token tile, 128 with more (a smaller activation tile)
    template <int MT> static constexpr int kb() { return MT == 1 ? 512 : 256; }
    static constexpr int kUpGroups = 1400;
    static constexpr int kKPerElem = 2;
};

constexpr int kPairRounds = APEX_MAX_PAIRS / kThreads;

// This thread's exec_idx entries, pairs r * 256 + t (the index clamped to P - 1; entries
// past P are dropped by expert_pairs).  Issued before a tile's first weight loads, so
// that the pair scan waits only for these, not for the weights.
__device__ __forceinline__ void pair_ids(const int32_t *__restrict__ exec_idx, int P,
                                         int (&ev)[kPairRounds]) {
#pragma unroll
    for (int r = 0; r < kPairRounds; ++r) {
        const int p = r * kThreads + threadIdx.x;
        ev[r] = exec_idx[p < P ? p : P - 1];
    }
}

// The pairs p < P with exec_idx[p] == e, in ascending order, into list[]; returns how
// many.  256 threads; P <= 1024 (four rounds of wave ballots).
__device__ int expert_pairs(const int (&ev)[kPairRounds], int P, int e, int *list,
                            int (*cnt)[4]) {
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    bool hit[kPairRounds];
    unsigned long long m[kPairRounds];
#pragma unroll
    for (int r = 0; r < kPairRounds; ++r) {
        hit[r] = r * kThreads + t < P && ev[r] == e;
        m[r] = __ballot(hit[r]);
        if (lane == 0) cnt[r][wave] = __popcll(m[r]);
    }
    __syncthreads();
    int base = 0;
#pragma unroll
    for (int r = 0; r < kPairRounds; ++r) {
        int off = base;
        for (int w = 0; w < wave; ++w) off += cnt[r][w];
        if (hit[r]) list[off + __popcll(m[r] & ((1ull << lane) - 1ull))] = r * kThreads + t;
        base += cnt[r][0] + cnt[r][1] + cnt[r][2] + cnt[r][3];
    }
    __syncthreads();
    return base;
}

// The K blocks of split z of a K range cut into blocks of kb values: nb blocks from b_lo,
// visited from a rotated start.  Workgroups start at different K blocks: tiles that run
// side by side then read different offsets of their rows instead of all hitting the same
// DRAM channels.
struct KBlocks {
    int b_lo, nb, rot, kb;
    __device__ __forceinline__ int k0(int b) const {
        const int q = b + rot;
        return (b_lo + (q >= nb ? q - nb : q)) * kb;
    }
};

__device__ __forceinline__ KBlocks k_blocks(int K, int kb, int splits, int z) {
    const int n = (K + kb - 1) / kb;
    KBlocks r;
    r.b_lo = z * n / splits;
    r.nb = (z + 1) * n / splits - r.b_lo;
    r.kb = kb;
    r.rot = int((blockIdx.x * 7u + blockIdx.y * 13u) % unsigned(r.nb > 0 ? r.nb : 1));
    return r;
}

// LDS of one workgroup's tile: bf16 weights and activations for bf16 slots; codes, MXFP4
// block scales and activations for the compact formats.  Rows are padded by 16
// bytes so that the 16 rows of a fragment read fall in distinct banks.
template <int NW, int MT, class WF, bool C = WF::kCodes>
struct GemmLds {
    uint16_t Ws[NW][kRows][kLdsRow];
    uint16_t Xs[16 * MT][kLdsRow];
};
template <int NW, int MT, class WF>
struct GemmLds<NW, MT, WF, true> {
    static constexpr int KB = WF::template kb<MT>();   // K values per block
    static constexpr int RB = KB / WF::kKPerElem;      // code bytes per row and block
    uint8_t Wc[NW][kRows][RB + 16];
    uint8_t Sc[NW][kRows][KB / 32];                    // MXFP4 block scales
    uint16_t Xs[16 * MT][KB + 8];
};

// 8 consecutive codes of row rr at K offset kc of the staged block, widened to bf16
// exactly (E4M3 values are bf16 values; an E2M1 value times its power-of-two scale too).
template <int NW, int MT, class WF>
__device__ __forceinline__ uint4 widen8(const GemmLds<NW, MT, WF, true> &lds, int m, int rr,
                                        int kc) {
    if constexpr (WF::kBlockScale) {
        const uint32_t c = *reinterpret_cast<const uint32_t *>(&lds.Wc[m][rr][kc / 2]);
        const float sc = apex::ffn::mx_scale(lds.Sc[m][rr][kc / 32]);
        return make_uint4(
            __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(c, sc, 0)),
            __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(c, sc, 1)),
            __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(c, sc, 2)),
            __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(c, sc, 3)));
    } else {
        const uint2 c = *reinterpret_cast<const uint2 *>(&lds.Wc[m][rr][kc]);
        const auto a = __builtin_amdgcn_cvt_pk_f32_fp8(int(c.x), false);
        const auto b = __builtin_amdgcn_cvt_pk_f32_fp8(int(c.x), true);
        const auto e = __builtin_amdgcn_cvt_pk_f32_fp8(int(c.y), false);
        const auto f = __builtin_amdgcn_cvt_pk_f32_fp8(int(c.y), true);
        const auto pk = [](float lo, float hi) {
            return (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xffff0000u);
        };
        return make_uint4(pk(a[0], a[1]), pk(b[0], b[1]), pk(e[0], e[1]), pk(f[0], f[1]));
    }
}

// One K block of a tile's weights in registers: every address valid (rows and K
// clamped), pieces outside the tile zeroed when the block is staged in LDS, not when it
// arrives, so that the loads stay in flight until then.
// bf16 slots: 16 threads per 256-byte piece of a row, 16 rows per pass of 256 threads.
template <int NW, int MT, class WF, bool C = WF::kCodes>
struct WRegs {
    static constexpr int kLoads = WBf16::kLoads, kRpp = WBf16::kRowsPerPass,
                         kTpr = WBf16::kThrPerRow;
    uint4 v[NW][kLoads];
    bool in = false;
    __device__ __forceinline__ void load(const uint16_t *const (&wbase)[NW], size_t wstride,
                                         const uint8_t *const (&)[NW], size_t, int rows_valid,
                                         int K, int k0) {
        const int t = threadIdx.x, wseg = t % kTpr, wr0 = t / kTpr;
        const int wk = k0 + 8 * wseg;
        in = wk < K;
        const int wkc = in ? wk : K - 8;
#pragma unroll
        for (int m = 0; m < NW; ++m)
#pragma unroll
            for (int j = 0; j < kLoads; ++j) {
                const int row = wr0 + kRpp * j;
                const int rc = row < rows_valid ? row : rows_valid - 1;
                v[m][j] = ld_stream(
                    reinterpret_cast<const uint4 *>(wbase[m] + size_t(rc) * wstride + wkc));
            }
    }
    __device__ __forceinline__ void stage(GemmLds<NW, MT, WF> &lds, int rows_valid) const {
        const int t = threadIdx.x, wseg = t % kTpr, wr0 = t / kTpr;
#pragma unroll
        for (int m = 0; m < NW; ++m)
#pragma unroll
            for (int j = 0; j < kLoads; ++j) {
                const int row = wr0 + kRpp * j;
                *reinterpret_cast<uint4 *>(&lds.Ws[m][row][8 * wseg]) =
                    keep_if(v[m][j], in && row < rows_valid);
            }
    }
};

// E4M3 and MXFP4 slots: the codes (and MXFP4 block scales) as stored, RB bytes per row
// and block.
template <int NW, int MT, class WF>
struct WRegs<NW, MT, WF, true> {
    using L = GemmLds<NW, MT, WF, true>;
    static constexpr int TPR = L::RB / 16;          // threads per row of a block
    static constexpr int RPP = kThreads / TPR;      // rows per pass
    static constexpr int NL = kRows / RPP;          // 16-byte loads per thread and matrix
    static constexpr int KPL = 16 * WF::kKPerElem;  // K values per 16-byte load
    uint4 v[NW][NL];
    uint32_t sc[NW][NL];
    bool in = false;
    __device__ __forceinline__ void load(const uint8_t *const (&wbase)[NW], size_t wstride,
                                         const uint8_t *const (&sbase)[NW], size_t sstride,
                                         int rows_valid, int K, int k0) {
        const int t = threadIdx.x, wseg = t % TPR, wr0 = t / TPR;
        const int wk = k0 + KPL * wseg;
        in = wk < K;
        const int wkc = in ? wk : K - KPL;
#pragma unroll
        for (int m = 0; m < NW; ++m)
#pragma unroll
            for (int j = 0; j < NL; ++j) {
                const int row = wr0 + RPP * j;
                const int rc = row < rows_valid ? row : rows_valid - 1;
                v[m][j] = ld_stream(reinterpret_cast<const uint4 *>(
                    wbase[m] + size_t(rc) * wstride + wkc / WF::kKPerElem));
                if constexpr (WF::kBlockScale) sc[m][j] = sbase[m][size_t(rc) * sstride + wkc / 32];
            }
    }
    __device__ __forceinline__ void stage(L &lds, int rows_valid) const {
        const int t = threadIdx.x, wseg = t % TPR, wr0 = t / TPR;
#pragma unroll
        for (int m = 0; m < NW; ++m)
#pragma unroll
            for (int j = 0; j < NL; ++j) {
                const int row = wr0 + RPP * j;
                *reinterpret_cast<uint4 *>(&lds.Wc[m][row][16 * wseg]) =
                    keep_if(v[m][j], in && row < rows_valid);
                if constexpr (WF::kBlockScale) lds.Sc[m][row][wseg] = uint8_t(sc[m][j]);
            }
    }
};

// Grouped-GEMM mainloop, shared by the gate/up and down projections and the weight
// formats.  A workgroup (4 wavefronts) owns a tile of 64 weight rows of NW weight
// matrices and up to 16*MT tokens, over the K blocks of kr.  Every thread loads 16-byte
// pieces so that each group of threads reads whole cache lines of one weight row, the
// block goes to LDS, and while the matrix cores work on it the next block is already
// loading into registers: every load address is valid (padding token rows read a real
// row), and zeroing and the fp32-to-bf16 conversion of activations happen at staging,
// so the first use of a loaded register comes after the matrix-core work on the previous
// block.  `w` may already hold the first block (w_ready): the kernels issue it before
// they look up the expert's pairs.
// bf16 slots: K blocks of kKB values as bf16 tiles.  E4M3 and MXFP4 slots: a block holds
// as many code bytes per row as a bf16 block (256 or 512 K values with one token tile,
// 128 or 256 with more), the codes go to LDS unchanged (the MXFP4 block scales beside
// them), and each wavefront widens its own fragments right before the matrix cores take
// them: every code is converted once, the bytes in flight per block match bf16, and the
// LDS moves a fraction of the widened data.
// Wavefront w multiplies its 16 rows with every token tile: v_mfma_f32_16x16x32_bf16,
// tokens as M, weight rows as N.  Tiles past the expert's last token multiply zero rows:
// skipping them on the token count made the compiler move the accumulators between
// register files around the skip, and the E4M3 kernel with two tiles then gave wrong
// sums that changed from run to run.
template <int NW, int MT, class Act, class WF>
__device__ __forceinline__ void gemm_tile(WRegs<NW, MT, WF> &w, bool w_ready,
                                          const typename WF::T *const (&wbase)[NW],
                                          size_t wstride, const uint8_t *const (&sbase)[NW],
                                          size_t sstride, int rows_valid, int K,
                                          const KBlocks &kr, const void *const (&xrow)[MT],
                                          const bool (&xok)[MT], GemmLds<NW, MT, WF> &lds,
                                          floatx4 (&acc)[NW][MT]) {
    constexpr int KB = WF::template kb<MT>();
    constexpr int QX = KB / 128;   // 8-value activation pieces per token row and thread
    const int t = threadIdx.x, wave = t / kWave, lane = t % kWave;
    const int seg = t & 15, r0 = t >> 4;
    typename Act::Raw xraw[QX][MT];
    bool x_in[QX];
#pragma unroll
    for (int m = 0; m < NW; ++m)
#pragma unroll
        for (int tt = 0; tt < MT; ++tt) acc[m][tt] = floatx4{0.f, 0.f, 0.f, 0.f};
    if (kr.nb <= 0) return;
    const auto load_x = [&](int k0) {
#pragma unroll
        for (int q = 0; q < QX; ++q) {
            const int kk = k0 + 128 * q + 8 * seg;
            x_in[q] = kk < K;
            const int kc = x_in[q] ? kk : K - 8;
#pragma unroll
            for (int j = 0; j < MT; ++j) xraw[q][j] = Act::load(xrow[j], kc);
        }
    };
    if (!w_ready) w.load(wbase, wstride, sbase, sstride, rows_valid, K, kr.k0(0));
    load_x(kr.k0(0));
    for (int b = 0; b < kr.nb; ++b) {
        __syncthreads();   // the previous block's fragments have been read
        w.stage(lds, rows_valid);
#pragma unroll
        for (int q = 0; q < QX; ++q)
#pragma unroll
            for (int j = 0; j < MT; ++j)
                *reinterpret_cast<uint4 *>(&lds.Xs[r0 + 16 * j][128 * q + 8 * seg]) =
                    keep_if(Act::to_bf16(xraw[q][j]), x_in[q] && xok[j]);
        __syncthreads();
        if (b + 1 < kr.nb) {
            w.load(wbase, wstride, sbase, sstride, rows_valid, K, kr.k0(b + 1));
            load_x(kr.k0(b + 1));
        }
        const int rr = 16 * wave + (lane & 15);
#pragma unroll 4
        for (int q = 0; q < KB / 32; ++q) {
            const int kc = 32 * q + 8 * (lane >> 4);
            uint4 wop[NW];
#pragma unroll
            for (int m = 0; m < NW; ++m) {
                if constexpr (WF::kCodes)
                    wop[m] = widen8(lds, m, rr, kc);
                else
                    wop[m] = *reinterpret_cast<const uint4 *>(&lds.Ws[m][rr][kc]);
            }
#pragma unroll
            for (int tt = 0; tt < MT; ++tt) {
                const uint4 xop = *reinterpret_cast<const uint4 *>(&lds.Xs[16 * tt + (lane & 15)][kc]);
#pragma unroll
                for (int m = 0; m < NW; ++m)
                    acc[m][tt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        as_bf16x8(xop), as_bf16x8(wop[m]), acc[m][tt], 0, 0, 0);
            }
        }
    }
}

// The fp32 row scales of an apex_pack_expert_fp8 slot: W1 rows, W3 rows, W2 rows.
template <class WF>
__device__ __forceinline__ const float *row_scales(const typename WF::T *slot, int d, int I) {
    return reinterpret_cast<const float *>(slot + size_t(3) * I * d);
}

// up_gemm: grid (ceil(I / 64), E, SU).  64 rows of W1 and W3 of expert blockIdx.y, every
// token of the expert (16*MT per pass), K blocks of split blockIdx.z.  slot_stride is
// the slot size in elements of WF::T.
// SU == 1: hb[pair, i] = bf16(silu(W1[i] . x_b) * (W3[i] . x_b)), ungated.
// SU  > 1: uv[(2z) * P*I + pair*I + i] = W1[i] . x_b over the split, uv[(2z+1) ...] = W3.
// E4M3 slots: the dot products are multiplied by the rows' scales.
template <int MT, int SU, class WF>
__global__ __launch_bounds__(kThreads) void up_gemm(
    const float *__restrict__ x, int d, int I, int P, int k, const int32_t *__restrict__ exec_idx,
    const int32_t *__restrict__ slot_of_expert, int n_slots,
    const typename WF::T *__restrict__ slots, size_t slot_stride, __bf16 *__restrict__ hb,
    float *__restrict__ uv) {
    __shared__ __align__(16) GemmLds<2, MT, WF> lds;
    __shared__ int list[APEX_MAX_PAIRS];
    __shared__ int cnt[kPairRounds][4];
    const int e = blockIdx.y;
    const int s = slot_of_expert[e];
    if (s < 0 || s >= n_slots) return;
    int ev[kPairRounds];
    pair_ids(exec_idx, P, ev);
    const int i0 = blockIdx.x * kRows;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const typename WF::T *slot = slots + size_t(s) * slot_stride;
    const typename WF::T *W = slot + size_t(i0) * 2 * d / WF::kKPerElem;
    const typename WF::T *const wbase[2] = {W, W + d / WF::kKPerElem};
    const size_t wstride = size_t(2) * d / WF::kKPerElem;
    // MXFP4 block scales of W1 and W3 rows i0.. (unused by the other formats)
    const uint8_t *sc = reinterpret_cast<const uint8_t *>(slot) + size_t(3) * I * d / 2;
    const uint8_t *const sbase[2] = {sc + size_t(i0) * (d / 32),
                                     sc + size_t(I + i0) * (d / 32)};
    const KBlocks kr = k_blocks(d, WF::template kb<MT>(), gridDim.z, blockIdx.z);
    // The first block's weights load while the expert's pairs are looked up, with no
    // branch in between (an empty split loads a clamped, valid block and drops it): at
    // the join after a branch the compiler would wait for the weights before the scan.
    WRegs<2, MT, WF> w;
    w.load(wbase, wstride, sbase, size_t(d / 32), I - i0, d, kr.k0(0));
    const int n_e = expert_pairs(ev, P, e, list, cnt);
    if (n_e == 0) return;
    for (int t0 = 0; t0 < n_e; t0 += 16 * MT) {
        const void *xrow[MT];
        bool xok[MT];
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            const int tok = t0 + (threadIdx.x >> 4) + 16 * j;
            xok[j] = tok < n_e;
            xrow[j] = x + size_t(list[xok[j] ? tok : 0] / k) * d;
        }
        floatx4 acc[2][MT];
        gemm_tile<2, MT, ActF32, WF>(w, t0 == 0, wbase, wstride, sbase, size_t(d / 32), I - i0,
                                     d, kr, xrow, xok, lds, acc);
        const int i = i0 + 16 * wave + (lane & 15);
        float s1 = 1.f, s3 = 1.f;
        if constexpr (WF::kFp8) {
            const float *sc = row_scales<WF>(slot, d, I);
            s1 = i < I ? sc[i] : 0.f;
            s3 = i < I ? sc[I + i] : 0.f;
        }
#pragma unroll
        for (int tt = 0; tt < MT; ++tt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int tok = t0 + 16 * tt + 4 * (lane >> 4) + r;
                if (tok < n_e && i < I) {
                    const size_t at = size_t(list[tok]) * I + i;
                    const float u = s1 * acc[0][tt][r], v = s3 * acc[1][tt][r];
                    if (SU == 1) {
                        hb[at] = (__bf16)(silu(u) * v);
                    } else {
                        uv[size_t(2 * blockIdx.z) * P * I + at] = u;
                        uv[size_t(2 * blockIdx.z + 1) * P * I + at] = v;
                    }
                }
            }
        __syncthreads();   // LDS is reused by the next pass
    }
}

// down_gemm: grid (ceil(d / 64), E, SD).  64 rows j of W2 of expert blockIdx.y, K (= I)
// blocks of split blockIdx.z.  yp[z * P*d + pair*d + j] = W2[j] . h[pair] over the split.
// The activations are the bf16 h rows.
template <int MT, class WF>
__global__ __launch_bounds__(kThreads) void down_gemm(
    int d, int I, int P, const int32_t *__restrict__ exec_idx,
    const int32_t *__restrict__ slot_of_expert, int n_slots,
    const typename WF::T *__restrict__ slots, size_t slot_stride, const __bf16 *__restrict__ hb,
    float *__restrict__ yp) {
    __shared__ __align__(16) GemmLds<1, MT, WF> lds;
    __shared__ int list[APEX_MAX_PAIRS];
    __shared__ int cnt[kPairRounds][4];
    const int e = blockIdx.y;
    const int s = slot_of_expert[e];
    if (s < 0 || s >= n_slots) return;
    int ev[kPairRounds];
    pair_ids(exec_idx, P, ev);
    const int j0 = blockIdx.x * kRows;
    const int wave = threadIdx.x / kWave, lane = threadIdx.x % kWave;
    const typename WF::T *slot = slots + size_t(s) * slot_stride;
    const typename WF::T *const wbase[1] = {
        slot + (size_t(2) * I * d + size_t(j0) * I) / WF::kKPerElem};
    const size_t wstride = size_t(I) / WF::kKPerElem;
    const uint8_t *const sbase[1] = {reinterpret_cast<const uint8_t *>(slot) +
                                     size_t(3) * I * d / 2 + size_t(2) * I * (d / 32) +
                                     size_t(j0) * (I / 32)};
    const KBlocks kr = k_blocks(I, WF::template kb<MT>(), gridDim.z, blockIdx.z);
    // the first block's weights load while the expert's pairs are looked up (as in up_gemm)
    WRegs<1, MT, WF> w;
    w.load(wbase, wstride, sbase, size_t(I / 32), d - j0, I, kr.k0(0));
    const int n_e = expert_pairs(ev, P, e, list, cnt);
    if (n_e == 0) return;
    float *out = yp + size_t(blockIdx.z) * P * d;
    for (int t0 = 0; t0 < n_e; t0 += 16 * MT) {
        const void *hrow[MT];
        bool hok[MT];
#pragma unroll
        for (int j = 0; j < MT; ++j) {
            const int tok = t0 + (threadIdx.x >> 4) + 16 * j;
            hok[j] = tok < n_e;
            hrow[j] = hb + size_t(list[hok[j] ? tok : 0]) * I;
        }
        floatx4 acc[1][MT];
        gemm_tile<1, MT, ActBf16, WF>(w, t0 == 0, wbase, wstride, sbase, size_t(I / 32), d - j0,
                                      I, kr, hrow, hok, lds, acc);
        const int j = j0 + 16 * wave + (lane & 15);
        float s2 = 1.f;
        if constexpr (WF::kFp8) s2 = j < d ? row_scales<WF>(slot, d, I)[2 * I + j] : 0.f;
#pragma unroll
        for (int tt = 0; tt < MT; ++tt)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int tok = t0 + 16 * tt + 4 * (lane >> 4) + r;
                if (tok < n_e && j < d)
                    out[size_t(list[tok]) * d + j] = s2 * acc[0][tt][r];
            }
        __syncthreads();   // LDS is reused by the next pass
    }
}

// swiglu_reduce: h[pair, i] = bf16(silu(sum_z u_z) * sum_z v_z) from up_gemm's SU split
// partials (splits added in order), for the pairs whose expert has a slot; 8 consecutive
// i per thread.
template <int SU>
__global__ __launch_bounds__(kThreads) void swiglu_reduce(
    int P, int I, int E, const int32_t *__restrict__ exec_idx,
    const int32_t *__restrict__ slot_of_expert, int n_slots, const float *__restrict__ uv,
    __bf16 *__restrict__ hb) {
    const int per = I / 8;
    const int g = blockIdx.x * kThreads + threadIdx.x;
    if (g >= P * per) return;
    const int p = g / per, i = 8 * (g - p * per);
    const int e = exec_idx[p];
    if (e < 0 || e >= E) return;
    const int sl = slot_of_expert[e];
    if (sl < 0 || sl >= n_slots) return;
    const size_t at = size_t(p) * I + i;
    *reinterpret_cast<uint4 *>(hb + at) = swiglu8<SU>(uv + at, size_t(P) * I);
}

// combine: y[b, j] (+)= sum over positions q of token b, in position order, of
// gate[q] * (sum over splits z, in order, of yp[z, pair, j]) for the pairs this pass
// executed.  Four consecutive j per thread.  Lane q of every wavefront looks up position
// q (its expert, slot and gate; k <= 64 since k <= E), so all positions cost one chain of
// dependent loads, and the wavefront reads them back with readlane.  The partial outputs
// of a group of positions are loaded before any is added (those of positions that were
// not executed are read and dropped).
template <int SD>
__global__ __launch_bounds__(kThreads) void combine_pairs(
    int B, int d, int E, int k, const int32_t *__restrict__ exec_idx,
    const float *__restrict__ exec_gate, const int32_t *__restrict__ slot_of_expert, int n_slots,
    const float *__restrict__ yp, float *__restrict__ y, int accumulate) {
    constexpr int kGroup = SD <= 2 ? 8 : 4;
    const int b = blockIdx.y;
    const int j = 4 * (blockIdx.x * kThreads + threadIdx.x);
    const int lane = threadIdx.x % kWave;
    int pos_ok = 0;
    float pos_gate = 0.f;
    if (lane < k) {
        const int p = b * k + lane;
        const int e = exec_idx[p];
        const bool e_ok = e >= 0 && e < E;
        const int sl = slot_of_expert[e_ok ? e : 0];
        pos_ok = e_ok && sl >= 0 && sl < n_slots;
        pos_gate = exec_gate[p];
    }
    if (j >= d) return;
    const size_t Pd = size_t(B) * k * d;
    const float *row = yp + size_t(b) * k * d + j;
    float4 *dst = reinterpret_cast<float4 *>(y + size_t(b) * d + j);
    const float4 o = *dst;   // read whether or not it is added, so no branch waits on it
    float4 s = make_float4(0.f, 0.f, 0.f, 0.f);
    const auto group = [&](int q0) {
        float4 v[kGroup][SD];
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
            const int q = min(q0 + u, k - 1);
#pragma unroll
            for (int z = 0; z < SD; ++z)
                v[u][z] = *reinterpret_cast<const float4 *>(row + z * Pd + size_t(q) * d);
        }
#pragma unroll
        for (int u = 0; u < kGroup; ++u) {
            if (q0 + u >= k) break;
            if (!__builtin_amdgcn_readlane(pos_ok, q0 + u)) continue;
            const float g = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(pos_gate), q0 + u));
            float4 t = v[u][0];
#pragma unroll
            for (int z = 1; z < SD; ++z) {
                t.x += v[u][z].x; t.y += v[u][z].y; t.z += v[u][z].z; t.w += v[u][z].w;
            }
            s.x += g * t.x; s.y += g * t.y; s.z += g * t.z; s.w += g * t.w;
        }
    };
    group(0);   // outside the loop, so its loads issue together with the read of y
    for (int q0 = kGroup; q0 < k; q0 += kGroup) group(q0);
    if (accumulate) s = make_float4(o.x + s.x, o.y + s.y, o.z + s.z, o.w + s.w);
    *dst = s;
}

// K splits of a projection with `groups` workgroups of work (row tiles times experts)
// and `nb` K blocks: `target` workgroups over all splits (rounded to the nearest split
// count when `nearest`, else up), at most kMaxSplit, and at least `min_blocks` K blocks
// per split.
int pick_splits(int groups, int nb, int target, bool nearest, int min_blocks) {
    groups = std::max(1, groups);
    int s = nearest ? (target + groups / 2) / groups : (target + groups - 1) / groups;
    s = std::min(s, kMaxSplit);
    s = std::min(s, std::max(1, nb / min_blocks));
    return std::max(s, 1);
}

struct Plan {
    int MT, SU, SD;
    size_t uv_bytes, h_bytes, y_bytes;   // h_bytes: the split partials (if any) and h
};

// The launch plan for weight format WF.  The split rules were fitted to timings of
// every split pair (1-4 each) on grouped calls of the Granite-3B, OLMoE, Mixtral,
// DeepSeek-16B and Phi-7B expert shapes in all three formats (24 to 64 resident
// experts): each K split adds a prologue (finding the expert's pairs, the first load)
// and partial sums, and pays only when the projection has too few workgroups to keep
// HBM busy.  The gate/up target grows with the per-byte cost of widening the codes
// (bf16 none, E4M3 most per byte); the down projection splits only over long K (for
// Mixtral's I = 14336).  The rule is within 1 % of the best split pair on average over
// those calls (the earlier rule, a common 1024-workgroup target with two K blocks per
// split, was 7 % off, and up to 25 % on OLMoE B64 with E4M3 experts).
template <class WF>
Plan plan_for(int B, int d, int I, int k, int E, int n_slots) {
    Plan pl;
    // token tiles per pass: enough for the whole batch on one expert up to 64 tokens
    pl.MT = B >= 48 ? 4 : (B >= 24 ? 2 : 1);
    const int experts = std::min(std::min(E, B * k), n_slots);
    const int kb = pl.MT == 4   ? WF::template kb<4>()
                   : pl.MT == 2 ? WF::template kb<2>()
                                : WF::template kb<1>();
    const int nb_d = (d + kb - 1) / kb, nb_i = (I + kb - 1) / kb;
    pl.SU = pick_splits((I + kRows - 1) / kRows * experts, nb_d, WF::kUpGroups, true, 3);
    pl.SD = pick_splits((d + kRows - 1) / kRows * experts, nb_i, 1024, false, 8);
    const size_t P = size_t(B) * k;
    pl.uv_bytes =
        pl.SU == 1 ? 0 : apex::align_up(size_t(2) * pl.SU * P * I * sizeof(float), 256);
    pl.h_bytes = pl.uv_bytes + P * I * 2;
    pl.y_bytes = size_t(pl.SD) * P * d * sizeof(float);
    return pl;
}

template <int MT, int SU, class WF>
void launch_up(dim3 g, hipStream_t st, const float *x, int d, int I, int P, int k,
               const int32_t *exec_idx, const int32_t *soe, int n_slots,
               const typename WF::T *slots, size_t stride, __bf16 *hb, float *uv) {
    hipLaunchKernelGGL((up_gemm<MT, SU, WF>), g, dim3(kThreads), 0, st, x, d, I, P, k, exec_idx,
                       soe, n_slots, slots, stride, hb, uv);
}

template <int MT, class WF>
void launch_up_splits(int SU, dim3 g, hipStream_t st, const float *x, int d, int I, int P, int k,
                      const int32_t *exec_idx, const int32_t *soe, int n_slots,
                      const typename WF::T *slots, size_t stride, __bf16 *hb, float *uv) {
    if (SU == 1)
        launch_up<MT, 1, WF>(g, st, x, d, I, P, k, exec_idx, soe, n_slots, slots, stride, hb, uv);
    else if (SU == 2)
        launch_up<MT, 2, WF>(g, st, x, d, I, P, k, exec_idx, soe, n_slots, slots, stride, hb, uv);
    else if (SU == 3)
        launch_up<MT, 3, WF>(g, st, x, d, I, P, k, exec_idx, soe, n_slots, slots, stride, hb, uv);
    else
        launch_up<MT, 4, WF>(g, st, x, d, I, P, k, exec_idx, soe, n_slots, slots, stride, hb, uv);
}

template <int MT, class WF>
void launch_down(dim3 g, hipStream_t st, int d, int I, int P, const int32_t *exec_idx,
                 const int32_t *soe, int n_slots, const typename WF::T *slots, size_t stride,
                 const __bf16 *hb, float *yp) {
    hipLaunchKernelGGL((down_gemm<MT, WF>), g, dim3(kThreads), 0, st, d, I, P, exec_idx, soe,
                       n_slots, slots, stride, hb, yp);
}

// The launches of one call for slots of weight format WF.
template <class WF>
apex_status run_grouped(const float *x, int B, int d, int I, int E, int k,
                        const int32_t *exec_idx, const float *exec_gate,
                        const int32_t *soe, const typename WF::T *slots, size_t stride,
                        int n_slots, float *y, int accumulate, char *wsb, hipStream_t stream) {
    const Plan pl = plan_for<WF>(B, d, I, k, E, n_slots);
    const int P = B * k;
    float *uv = reinterpret_cast<float *>(wsb);
    __bf16 *hb = reinterpret_cast<__bf16 *>(wsb + pl.uv_bytes);
    float *yp = reinterpret_cast<float *>(wsb + apex::align_up(pl.h_bytes, 256));
    const dim3 gu((I + kRows - 1) / kRows, E, pl.SU);
    if (pl.MT == 4)
        launch_up_splits<4, WF>(pl.SU, gu, stream, x, d, I, P, k, exec_idx, soe, n_slots, slots,
                                stride, hb, uv);
    else if (pl.MT == 2)
        launch_up_splits<2, WF>(pl.SU, gu, stream, x, d, I, P, k, exec_idx, soe, n_slots, slots,
                                stride, hb, uv);
    else
        launch_up_splits<1, WF>(pl.SU, gu, stream, x, d, I, P, k, exec_idx, soe, n_slots, slots,
                                stride, hb, uv);
    APEX_HIP(hipGetLastError());
    if (pl.SU > 1) {
        const dim3 gr((P * (I / 8) + kThreads - 1) / kThreads);
        if (pl.SU == 2)
            hipLaunchKernelGGL(swiglu_reduce<2>, gr, dim3(kThreads), 0, stream, P, I, E, exec_idx,
                               soe, n_slots, uv, hb);
        else if (pl.SU == 3)
            hipLaunchKernelGGL(swiglu_reduce<3>, gr, dim3(kThreads), 0, stream, P, I, E, exec_idx,
                               soe, n_slots, uv, hb);
        else
            hipLaunchKernelGGL(swiglu_reduce<4>, gr, dim3(kThreads), 0, stream, P, I, E, exec_idx,
                               soe, n_slots, uv, hb);
        APEX_HIP(hipGetLastError());
    }

    const dim3 gd((d + kRows - 1) / kRows, E, pl.SD);
    if (pl.MT == 4)
        launch_down<4, WF>(gd, stream, d, I, P, exec_idx, soe, n_slots, slots, stride, hb, yp);
    else if (pl.MT == 2)
        launch_down<2, WF>(gd, stream, d, I, P, exec_idx, soe, n_slots, slots, stride, hb, yp);
    else
        launch_down<1, WF>(gd, stream, d, I, P, exec_idx, soe, n_slots, slots, stride, hb, yp);
    APEX_HIP(hipGetLastError());
    const dim3 gc((d / 4 + kThreads - 1) / kThreads, B);
    if (pl.SD == 1)
        hipLaunchKernelGGL(combine_pairs<1>, gc, dim3(kThreads), 0, stream, B, d, E, k, exec_idx,
                           exec_gate, soe, n_slots, yp, y, accumulate);
    else if (pl.SD == 2)
        hipLaunchKernelGGL(combine_pairs<2>, gc, dim3(kThreads), 0, stream, B, d, E, k, exec_idx,
                           exec_gate, soe, n_slots, yp, y, accumulate);
    else if (pl.SD == 3)
        hipLaunchKernelGGL(combine_pairs<3>, gc, dim3(kThreads), 0, stream, B, d, E, k, exec_idx,
                           exec_gate, soe, n_slots, yp, y, accumulate);
    else
        hipLaunchKernelGGL(combine_pairs<4>, gc, dim3(kThreads), 0, stream, B, d, E, k, exec_idx,
                           exec_gate, soe, n_slots, yp, y, accumulate);
    APEX_HIP(hipGetLastError());
    return APEX_OK;
}

}  // namespace

namespace apex {

// [2*SU fp32 split partials, when SU > 1][h: bf16 B*k x I][per-split, per-pair outputs:
//  SD x B*k x d fp32]
size_t ffn_grouped_workspace(int B, int d, int I, int k) {
    // the largest plan over the slot counts and weight formats the call can be given
    size_t worst = 0;
    const auto cover = [&](const Plan &pl) {
        worst = std::max(worst, align_up(pl.h_bytes, 256) + align_up(pl.y_bytes, 256));
    };
    for (int experts = 1; experts <= APEX_MAX_EXPERTS; ++experts) {
        cover(plan_for<WBf16>(B, d, I, k, APEX_MAX_EXPERTS, experts));
        cover(plan_for<WE4M3>(B, d, I, k, APEX_MAX_EXPERTS, experts));
        cover(plan_for<WMxfp4>(B, d, I, k, APEX_MAX_EXPERTS, experts));
    }
    return worst;
}

void ffn_grouped_plan(int B, int d, int I, int E, int k, int n_slots, WeightFormat fmt,
                      int32_t out[3]) {
    const Plan pl = fmt == WeightFormat::kE4M3    ? plan_for<WE4M3>(B, d, I, k, E, n_slots)
                    : fmt == WeightFormat::kMxfp4 ? plan_for<WMxfp4>(B, d, I, k, E, n_slots)
                                                  : plan_for<WBf16>(B, d, I, k, E, n_slots);
    out[0] = pl.MT;
    out[1] = pl.SU;
    out[2] = pl.SD;
}

apex_status ffn_grouped(const float *x, int B, int d, int I, int E, int k,
                        const int32_t *exec_idx, const float *exec_gate,
                        const int32_t *slot_of_expert, const void *slots, int n_slots,
                        WeightFormat fmt, float *y, int accumulate, void *workspace,
                        hipStream_t stream) {
    char *wsb = static_cast<char *>(workspace);
    if (fmt == WeightFormat::kE4M3)
        return run_grouped<WE4M3>(x, B, d, I, E, k, exec_idx, exec_gate, slot_of_expert,
                                  static_cast<const uint8_t *>(slots),
                                  apex_expert_bytes_fp8(d, I), n_slots, y, accumulate, wsb,
                                  stream);
    if (fmt == WeightFormat::kMxfp4)
        return run_grouped<WMxfp4>(x, B, d, I, E, k, exec_idx, exec_gate, slot_of_expert,
                                   static_cast<const uint8_t *>(slots),
                                   apex_expert_bytes_mxfp4(d, I), n_slots, y, accumulate, wsb,
                                   stream);
    return run_grouped<WBf16>(x, B, d, I, E, k, exec_idx, exec_gate, slot_of_expert,
                              static_cast<const uint16_t *>(slots), size_t(3) * d * I, n_slots,
                              y, accumulate, wsb, stream);
}

}  // namespace apex
