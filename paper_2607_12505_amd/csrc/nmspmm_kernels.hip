// GEMM kernels of libnmspmm for gfx950 (CDNA4): Y = X W^T in int8 with int32
// accumulation, optional per-channel fp16 dequantisation and int8
// requantisation; and the binary16 -> int8 activation quantiser.
//
// Orientation: the weight is the A operand and the activations the B operand
// of the matrix instruction, so a 16 x 16 accumulator holds 16 output channels
// x 16 tokens.  This orientation is forced by the structured-sparse
// instruction, whose sparse operand is A.
//
// Dataflow of one workgroup (4 or 8 waves) over its k range, one 128-wide
// k-step at a time (paper Sec. 4.2: sparse handling confined to packed
// loading, the compute stage purely matrix-instruction based):
//   - every X byte reaches LDS through the direct-to-LDS 16-byte loads of
//     gfx950, into a ring of NST k-step slots filled NST-1 steps ahead of the
//     compute: the tile_m x 128 slice of X, and with it the weight slice as
//     stored when it is already what the matrix instruction reads (the 4:2
//     fragments of 2:4, or tile_n x 128 rows of a dense W).  Each workgroup
//     fetches each byte once; no VGPRs are spent on staging, so the ring
//     depth costs only LDS.  Each lane picks the source chunk that belongs at
//     its LDS slot, so row-major slices land with their 16-byte chunks
//     XOR-swizzled by row and the operand reads of 16 rows hit distinct banks;
//   - compact weights (1:4, 1:8, 2:8 and the 3:8-5:8 mask layouts) are
//     expanded on the way (Sec. 4.2): in k_gemm each wave loads its blocks of
//     the next k-step into registers and writes them, expanded, into the slot
//     (the 4:2 operand or swizzled dense rows); in k_gemm_ks the 1:4, 1:8 and
//     2:8 blocks travel through the ring like X and are expanded straight into
//     the operand registers.  k_expand does the same expansion once per call
//     into the workspace when the planner prefers that;
//   - the loads are issued from inline assembly and their completion is
//     awaited explicitly (vector-memory counter, then one barrier per k-step),
//     so the compiler does not serialise the ring with conservative waits;
//   - each wave runs FN x FM accumulators: per k-step it reads its FN weight
//     fragments from LDS once, then per token fragment the B operand once,
//     reused by all FN weight fragments;
//   - the epilogue goes back through LDS, 16 tokens at a time, so that every
//     store instruction writes whole rows of the wave's tile: 16 lanes cover
//     256 contiguous bytes of int32 (128 of fp16, 64 of int8) per token;
//   - split-K (Sec. 4.3): every split runs the same code on its k range and
//     stores its int32 partial tile; the last split to arrive at a tile
//     (atomic counter) adds the partials and runs the epilogue, so merging
//     happens once, at the end.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "nmspmm_internal.h"

namespace nmspmm {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef unsigned short v4u16 __attribute__((ext_vector_type(4)));

// Workgroups are dispatched round-robin over the 8 XCDs (each with its own
// L2).  Renumber them so that consecutive logical tiles -- which share the
// same rows of X -- run on the same XCD.
__device__ inline int map_block(int bid, int nwg) {
    const int xcd = bid & 7, local = bid >> 3;
    const int per = nwg >> 3, rem = nwg & 7;
    return xcd < rem ? xcd * (per + 1) + local : rem * (per + 1) + (xcd - rem) * per + local;
}

// Logical tile -> (column tile tn, row index `rest`) over `rows` rows of
// tiles_n tiles.  group_rows == 0: row by row (consecutive tiles share rows of
// X and sweep all of W).  Otherwise groups of group_rows rows, each walked
// column by column, so the tiles in flight on one XCD touch a group's rows of
// X and only part of W.  Either way a bijection onto [0, rows * tiles_n).
__device__ inline void tile_order(int lid, int tiles_n, int rows, int group_rows, int *tn, int *rest) {
    if (group_rows <= 0) {
        *tn = lid % tiles_n;
        *rest = lid / tiles_n;
        return;
    }
    const int span = group_rows * tiles_n;
    const int g = lid / span, r = lid - g * span;
    const int left = rows - g * group_rows;
    const int h = left < group_rows ? left : group_rows;
    *rest = g * group_rows + r % h;
    *tn = r / h;
}

// Buffer-resource word 3 for raw 32-bit accesses, and the cache-policy bit
// that makes a buffer access coherent at agent scope (sc1).
constexpr int kBufferFlags = 0x00020000;
constexpr int kSc1 = 16;
// Cache policy of the output stores: non-temporal.  Timed inside whole
// workload steps (every GEMM's buffers evicted by the others' traffic before
// it runs again), streaming the outputs past L2 and the last-level cache beat
// the default and the device-scope (sc1) policies on every workload, by up to
// a third on outputs larger than the 256 MB last-level cache.
constexpr int kStoreNT = 2;

// Direct-to-LDS loads: lane L's bytes land at lds_base + L * size.  lds_base
// must be wave-uniform (it goes through M0).  M0 is a register the compiler
// reserves, so it warns that the clobber below may not be honoured; the
// generated code of these kernels uses M0 nowhere else (LDS instructions do
// not need it on gfx950), so nothing live is overwritten.
__device__ inline void dma16(const void *g, uint32_t lds_base) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "s"(lds_base) : "memory", "m0");
}
__device__ inline void dma4(const void *g, uint32_t lds_base) {
    asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" ::"v"(g), "s"(lds_base) : "memory", "m0");
}
// The same with a wave-uniform 64-bit base in SGPRs and a 32-bit per-lane
// byte offset: no per-lane 64-bit address arithmetic.
__device__ inline void dma16o(const void *base, uint32_t off, uint32_t lds_base) {
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "s"(lds_base)
                 : "memory", "m0");
}
__device__ inline void dma4o(const void *base, uint32_t off, uint32_t lds_base) {
    asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dword %0, %1" ::"v"(off), "s"(base), "s"(lds_base)
                 : "memory", "m0");
}

// Wait until at most N of this wave's vector-memory operations are in flight
// and all of its LDS operations are done, then the workgroup barrier.
template <int N>
__device__ inline void wait_then_barrier() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4));
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// Wait (no barrier) until at most N of this wave's vector-memory operations
// are in flight and all of its LDS operations are done.
template <int N>
__device__ inline void wait_only() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4));
    asm volatile("" ::: "memory");
}

template <int L, int DMA>
__device__ inline void wait_later(int later) {
    if constexpr (L <= 0) {
        wait_only<0>();
    } else {
        if (later >= L) {
            constexpr int n = L * DMA <= 63 ? L * DMA : (63 / DMA) * DMA;
            wait_only<n>();
        } else {
            wait_later<L - 1, DMA>(later);
        }
    }
}

// Barrier of k-step iteration with `later` k-steps (each DMA loads per wave)
// still allowed in flight: dispatches to the matching immediate.  The vmcnt
// field holds at most 63; beyond that fewer loads are allowed in flight
// (waiting longer is always safe).
template <int L, int DMA>
__device__ inline void wait_later_then_barrier(int later) {
    if constexpr (L <= 0) {
        wait_then_barrier<0>();
    } else {
        if (later >= L) {
            constexpr int n = L * DMA <= 63 ? L * DMA : (63 / DMA) * DMA;
            wait_then_barrier<n>();
        } else {
            wait_later_then_barrier<L - 1, DMA>(later);
        }
    }
}

// int8 code of a binary32 value: nearest integer (ties to even), saturated
// to [-127, 127], NaN -> 0.
__device__ inline int q8(float v) {
    if (v != v) return 0;
    const float r = __builtin_rintf(v);
    return (int)fminf(fmaxf(r, -127.0f), 127.0f);
}

// Per-channel multipliers of the epilogue outputs for 4 consecutive channels.
struct EpiScale {
    v4f sc;   // dequantisation (fp16 output)
    v4f qs;   // requantisation (int8 output)
};

typedef unsigned int v2u __attribute__((ext_vector_type(2)));
typedef unsigned int v4u __attribute__((ext_vector_type(4)));

// Writes 4 consecutive channels of one token: int32, fp16(fp32(y) * scale)
// and/or the int8 code q8(fp32(y) * qscale), whichever outputs are present.
// Buffer stores with a 32-bit element offset (outputs hold fewer than 2^29
// elements, checked on the host): the per-lane address is one 32-bit
// multiply-add instead of 64-bit pointer arithmetic, and the hardware drops
// any write past the end of an output.
__device__ inline void emit_out(const GemmArgs &a, int tok, int ch, const v4i &v, const EpiScale &es) {
    const uint32_t e = (uint32_t)tok * (uint32_t)a.n + (uint32_t)ch;
    const uint32_t elems = (uint32_t)a.m * (uint32_t)a.n;
    if (a.Y) {
        const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(a.Y, 0, (int)(elems * 4), kBufferFlags);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, v), r, (int)(e * 4), 0, kStoreNT);
    }
    if (a.Yh) {
        v4u16 h;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const _Float16 x = (_Float16)((float)v[i] * es.sc[i]);
            h[i] = __builtin_bit_cast(unsigned short, x);
        }
        const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(a.Yh, 0, (int)(elems * 2), kBufferFlags);
        __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(v2u, h), r, (int)(e * 2), 0, kStoreNT);
    }
    if (a.Yq) {
        uint32_t packed = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) packed |= (uint32_t)(q8((float)v[i] * es.qs[i]) & 0xFF) << (8 * i);
        const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(a.Yq, 0, (int)elems, kBufferFlags);
        __builtin_amdgcn_raw_buffer_store_b32(packed, r, (int)e, 0, kStoreNT);
    }
}

// Multipliers read in place of an absent multiplier array (the value is never
// used: the output it scales is absent too).  A valid address owned by the
// library, so no caller pointer is read for a missing array.
__device__ const float kNoScale[4] = {1.0f, 1.0f, 1.0f, 1.0f};

// The multipliers of 4 consecutive channels.  The loads are issued whatever
// outputs are present (from kNoScale when a multiplier array is absent, or
// from channel 0 past n) so that no branch guards them: the compiler then
// waits for them once, at their first use, instead of emitting a full
// vector-memory wait before every later use, which would also wait for every
// store issued in between.
//
// The loads are also awaited right away (all vector-memory operations of the
// wave): the compiler's own wait tracking cannot see through the output
// branches of emit_out and would otherwise wait again before every store.
// Callers load the multipliers where nothing else of theirs is in flight
// that they could keep waiting for.
__device__ inline EpiScale load_scale(const GemmArgs &a, int ch) {
    const int c = ch < a.n ? ch : 0;
    const float *sc = a.scale ? a.scale + c : kNoScale;
    const float *qs = a.qscale ? a.qscale + c : kNoScale;
    EpiScale es;
    es.sc = *(const v4f *)sc;
    es.qs = *(const v4f *)qs;
    __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0); expcnt and lgkmcnt not waited for
    return es;
}

// Split-K partial sums: [split_k x m x n] int32 below 2 GiB (checked by the
// planner), accessed with agent-coherent (sc1) buffer operations: visible to
// every XCD once complete, with no write-back of the non-coherent L2 needed.
__device__ inline __amdgpu_buffer_rsrc_t partial_rsrc(const GemmArgs &a) {
    return __builtin_amdgcn_make_buffer_rsrc(a.partials, 0, a.split_k > 1 ? a.split_k * a.m * a.n * 4 : 0,
                                             kBufferFlags);
}

__device__ inline void publish_partial(const GemmArgs &a, __amdgpu_buffer_rsrc_t r, int split, int tok, int ch,
                                       const v4i &v) {
    __builtin_amdgcn_raw_buffer_store_b128(v, r, ((split * a.m + tok) * a.n + ch) << 2, 0, kSc1);
}

__device__ inline v4i merge_partials(const GemmArgs &a, __amdgpu_buffer_rsrc_t r, int tok, int ch) {
    v4i sum = v4i{0, 0, 0, 0};
    for (int sp = 0; sp < a.split_k; ++sp)
        sum += __builtin_amdgcn_raw_buffer_load_b128(r, ((sp * a.m + tok) * a.n + ch) << 2, 0, kSc1);
    return sum;
}

// After every thread published its part of this split's partial tile: count
// the arrival and tell whether this workgroup is the last split of the tile
// (then it merges).  Ordering: the barrier makes every wave's partial stores
// happen before thread 0's arrival, which is a release at agent scope, so a
// split that arrives later and reads the count with acquire ordering sees
// them; the last arriver's acquire is passed to its other threads by the
// second barrier.  (The wait for this wave's stores before the barrier is
// not needed by that argument; it keeps the stores complete before the
// counter moves.)  The counter is left at zero for the next call.
__device__ inline bool arrive_last(const GemmArgs &a, int tile, int *s_flag) {
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (threadIdx.x == 0) {
        const int old = __hip_atomic_fetch_add(&a.counters[tile], 1, __ATOMIC_ACQ_REL, __HIP_MEMORY_SCOPE_AGENT);
        const int last = old == a.split_k - 1;
        if (last) __hip_atomic_store(&a.counters[tile], 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        *s_flag = last;
    }
    __syncthreads();
    return *s_flag != 0;
}

// ---------------------------------------------------------------------------
// Weight kinds.  The weight reaches LDS either as stored (DMA: the 4:2 operand
// of 2:4, or plain rows of a dense W) or in a compact packed form that every
// workgroup loads into registers one k-step ahead, expands, and writes to LDS
// in the form the matrix instruction reads (paper Sec. 4.2: decoding
// overlapped with shared-memory placement and matrix issue): the 4:2 operand
// for 1:4, 1:8 and 2:8, a dense tile for the mask layouts of 3:8, 4:8 and 5:8.
// (The k-sliced kernel instead stages the 1:4, 1:8 and 2:8 blocks in its ring
// as stored and expands them into operand registers, see k_gemm_ks.)

template <int KIND>
struct Kind {
    static constexpr bool kSp = kind_is_sp42(KIND);                         // smfmac on the 4:2 operand
    static constexpr bool kDecode = KIND != NM_KIND_SP42 && KIND != NM_KIND_DENSE;
    static constexpr int VB = KIND == NM_KIND_DENSE ? 0 : layout_lane_vbytes(KIND);  // value bytes per lane
    static constexpr int MB = KIND == NM_KIND_DENSE ? 0 : layout_lane_mbytes(KIND);  // position bytes per lane
    static constexpr int NV = layout_mask_values(KIND);                     // values per window (mask layouts)
    static constexpr int VW = VB / 4 > 0 ? VB / 4 : 1;                       // value dwords per lane
    // vector-memory loads per lane and block (as wload issues them): values
    // (one vector for 8 and 16 bytes, else one per dword) and positions
    static constexpr int LOADS = !kDecode ? 0 : (VB == 8 || VB == 16 ? 1 : VB / 4) + 1;
    // LDS lookup table: 2:8 position codes (64) and window masks (256)
    static constexpr int LUT = KIND == NM_KIND_C28 ? 64 : NV > 0 ? 256 : 1;
};

// One lane's compact bytes of one block, in registers.
template <int KIND>
struct WRegs {
    uint32_t v[Kind<KIND>::VW];
    uint32_t m;
};

// Lane values sit at L * VB bytes of a 16-byte aligned block: 8 and 16 bytes
// per lane keep 8- and 16-byte alignment and load as one vector; 4, 12 and 20
// bytes are only 4-byte aligned and load as dwords (never as a wider vector,
// which could read past the end of the buffer).
template <int KIND>
__device__ __forceinline__ void wload(WRegs<KIND> &r, const int8_t *vals, const uint8_t *meta) {
    constexpr int VB = Kind<KIND>::VB;
    if constexpr (VB == 8) {
        const v2u t = *(const v2u *)vals;
        r.v[0] = t[0];
        r.v[1] = t[1];
    } else if constexpr (VB == 16) {
        const v4u t = *(const v4u *)vals;
#pragma unroll
        for (int i = 0; i < 4; ++i) r.v[i] = t[i];
    } else {
        static_assert(VB % 4 == 0 && VB <= 20, "value bytes per lane");
#pragma unroll
        for (int i = 0; i < VB / 4; ++i) r.v[i] = ((const uint32_t *)vals)[i];
    }
    if constexpr (Kind<KIND>::MB == 2)
        r.m = *(const uint16_t *)meta;
    else
        r.m = *(const uint32_t *)meta;
}

// 2:8 table: position code c = o0 | o1 << 3 of a window (its two slots) ->
// {byte selector placing the window's two values (source bytes 0 and 1) in
// the 4:2 slots of its two 4-groups, position byte of those groups}.  Both
// slots in one half: that group takes them in order, the other group holds
// zeros at the same positions; one slot per half: each group takes its value
// in slot 0 and a zero at the position next to it (p ^ 1) in slot 1.
__device__ inline uint2 c28_entry(int c) {
    const int o0 = c & 7, o1 = c >> 3;
    const int h0 = o0 >> 2, h1 = o1 >> 2, p0 = o0 & 3, p1 = o1 & 3;
    uint32_t sel = 0x0C0C0C0Cu, ib;
    if (h0 == h1) {
        sel = (sel & ~(0xFFFFu << (16 * h0))) | (0x0100u << (16 * h0));
        const uint32_t nib = (uint32_t)(p0 | (p1 << 2));
        ib = nib | (nib << 4);
    } else {
        sel = (sel & ~(0xFFu << (16 * h0))) | (0x00u << (16 * h0));
        sel = (sel & ~(0xFFu << (16 * h1))) | (0x01u << (16 * h1));
        ib = ((uint32_t)(p0 | ((p0 ^ 1) << 2)) << (4 * h0)) | ((uint32_t)(p1 | ((p1 ^ 1) << 2)) << (4 * h1));
    }
    return uint2{sel, ib};
}

// Mask table: window mask mu -> byte selectors of its 8 positions (low and
// high 4): the rank of the position among the set bits (which source byte
// holds its value) for a set bit, the zero selector 0x0C otherwise.
__device__ inline uint2 mask_entry(int mu) {
    uint32_t s[2] = {0, 0};
    int rank = 0;
    for (int p = 0; p < 8; ++p) {
        const uint32_t b = ((mu >> p) & 1) ? (uint32_t)rank++ : 0x0Cu;
        s[p >> 2] |= b << (8 * (p & 3));
    }
    return uint2{s[0], s[1]};
}

template <int KIND>
__device__ inline void fill_lut(uint2 *lut, int tid, int nthreads) {
    if constexpr (KIND == NM_KIND_C28) {
        for (int e = tid; e < 64; e += nthreads) lut[e] = c28_entry(e);
    } else if constexpr (Kind<KIND>::NV > 0) {
        for (int e = tid; e < 256; e += nthreads) lut[e] = mask_entry(e);
    }
}

// Expands one lane's compact block into its 4:2 operand: 16 value bytes
// (two slots per 4-group) and the position word (nibble g: slot 0 position,
// slot 1 position << 2).
template <int KIND>
__device__ __forceinline__ void expand_sp42(const WRegs<KIND> &r, const uint2 *lut, v4i &vals, uint32_t &idx) {
    if constexpr (KIND == NM_KIND_C14) {
        // group g: its value in slot 0 at position o, a zero in slot 1 at o ^ 1
        vals[0] = (int)__builtin_amdgcn_perm(r.v[1], r.v[0], 0x0C010C00u);
        vals[1] = (int)__builtin_amdgcn_perm(r.v[1], r.v[0], 0x0C030C02u);
        vals[2] = (int)__builtin_amdgcn_perm(r.v[1], r.v[0], 0x0C050C04u);
        vals[3] = (int)__builtin_amdgcn_perm(r.v[1], r.v[0], 0x0C070C06u);
        uint32_t x = r.m;                               // 2-bit positions -> one per nibble
        x = (x | (x << 8)) & 0x00FF00FFu;
        x = (x | (x << 4)) & 0x0F0F0F0Fu;
        x = (x | (x << 2)) & 0x33333333u;
        idx = x | ((x ^ 0x11111111u) << 2);
    } else if constexpr (KIND == NM_KIND_C18) {
        // window w: 3-bit position o = 4 h + p -> byte w of ob; its value goes
        // to slot 0 of group h (byte 2 h of the window's dword) at position p,
        // a zero at p ^ 1; the empty group holds zeros at the same positions
        uint32_t x = (r.m & 0x3Fu) | ((r.m & 0xFC0u) << 10);
        const uint32_t ob = (x & 0x00070007u) | ((x & 0x00380038u) << 5);
        idx = __builtin_amdgcn_perm(0xBBEE1144u, 0xBBEE1144u, ob);   // byte: (p | (p ^ 1) << 2) * 0x11
        const uint32_t sh = (ob & 0x04040404u) << 2;                  // byte w: 16 h
#pragma unroll
        for (int w = 0; w < 4; ++w)
            vals[w] = (int)(__builtin_amdgcn_perm(0u, r.v[0], 0x0C0C0C00u | (uint32_t)w) << ((sh >> (8 * w)) & 16u));
    } else {
        static_assert(KIND == NM_KIND_C28, "4:2 expansion");
        idx = 0;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            const uint2 e = lut[(r.m >> (6 * w)) & 63u];
            const uint32_t src = r.v[w >> 1] >> (16 * (w & 1));     // the window's two values in bytes 0, 1
            vals[w] = (int)__builtin_amdgcn_perm(0u, src, e.x);
            idx |= e.y << (8 * w);
        }
    }
}

// Expands one lane's mask-layout block into its 32 dense weights (two
// 16-byte chunks: windows 0-1 and 2-3).
template <int KIND>
__device__ __forceinline__ void expand_dense(const WRegs<KIND> &r, const uint2 *lut, v4i &c0, v4i &c1) {
    constexpr int NV = Kind<KIND>::NV, VW = Kind<KIND>::VW;
    uint32_t out[8];
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        const int b = NV * w;                                    // first value byte of the window
        const uint32_t d0 = r.v[b / 4];
        const uint32_t d1 = b / 4 + 1 < VW ? r.v[b / 4 + 1] : 0u;
        const uint32_t d2 = b / 4 + 2 < VW ? r.v[b / 4 + 2] : 0u;
        const uint32_t lo = __builtin_amdgcn_alignbyte(d1, d0, (uint32_t)(b % 4));   // bytes b .. b+3
        const uint32_t hi = __builtin_amdgcn_alignbyte(d2, d1, (uint32_t)(b % 4));   // bytes b+4 .. b+7
        const uint2 e = lut[(r.m >> (8 * w)) & 0xFFu];
        out[2 * w] = __builtin_amdgcn_perm(hi, lo, e.x);
        out[2 * w + 1] = __builtin_amdgcn_perm(hi, lo, e.y);
    }
    c0 = v4i{(int)out[0], (int)out[1], (int)out[2], (int)out[3]};
    c1 = v4i{(int)out[4], (int)out[5], (int)out[6], (int)out[7]};
}

// Expands lane `lane`'s part of a compact block and writes it to the LDS
// weight area of a slot: block bl of the tile (16 rows), in the layout the
// compute stage reads (4:2 operand, or swizzled dense rows).
template <int KIND, int WVB>
__device__ __forceinline__ void expand_to_lds(const WRegs<KIND> &r, const uint2 *lut, int8_t *wslot, int bl,
                                              int lane) {
    if constexpr (Kind<KIND>::kSp) {
        v4i vals;
        uint32_t idx;
        expand_sp42<KIND>(r, lut, vals, idx);
        *(v4i *)(wslot + bl * kVBlock + lane * 16) = vals;
        *(uint32_t *)(wslot + WVB + bl * kMBlock + lane * 4) = idx;
    } else {
        v4i c0, c1;
        expand_dense<KIND>(r, lut, c0, c1);
        const int row = bl * 16 + (lane & 15);
        const int ch = 2 * (lane >> 4);                          // the lane's first 16-byte chunk of the row
        int8_t *rowp = wslot + row * 128;
        *(v4i *)(rowp + ((ch ^ (row & 7)) << 4)) = c0;
        *(v4i *)(rowp + (((ch + 1) ^ (row & 7)) << 4)) = c1;
    }
}

// A workgroup past the GEMM's own (blockIdx.x >= gemm_grid) expands blocks
// of another compact weight, one per wave, with its lookup table in the
// GEMM's LDS (at least 2 KB): so a launch can carry the expansion a later
// GEMM needs without a launch of its own.
template <int KIND>
__device__ __forceinline__ void expand_block(const int8_t *__restrict__ vals, const uint8_t *__restrict__ meta, int n,
                                             int k, int blocks, int k_steps, int8_t *out, int b, int lane, uint2 *lut,
                                             int tid, int nthreads);

__device__ inline void expand_tail(const GemmArgs &a, uint2 *lut) {
    const int tid = threadIdx.x, nthreads = blockDim.x;
    const int b = ((int)blockIdx.x - a.gemm_grid) * (nthreads >> 6) + (tid >> 6), lane = tid & 63;
    switch (a.x_kind) {
        case NM_KIND_C14:
            expand_block<NM_KIND_C14>(a.x_vals, a.x_meta, a.x_n, a.x_k, a.x_blocks, a.x_k_steps, a.x_out, b, lane, lut,
                                      tid, nthreads);
            break;
        case NM_KIND_C18:
            expand_block<NM_KIND_C18>(a.x_vals, a.x_meta, a.x_n, a.x_k, a.x_blocks, a.x_k_steps, a.x_out, b, lane, lut,
                                      tid, nthreads);
            break;
        case NM_KIND_C28:
            expand_block<NM_KIND_C28>(a.x_vals, a.x_meta, a.x_n, a.x_k, a.x_blocks, a.x_k_steps, a.x_out, b, lane, lut,
                                      tid, nthreads);
            break;
        case NM_KIND_MK3:
            expand_block<NM_KIND_MK3>(a.x_vals, a.x_meta, a.x_n, a.x_k, a.x_blocks, a.x_k_steps, a.x_out, b, lane, lut,
                                      tid, nthreads);
            break;
        case NM_KIND_MK4:
            expand_block<NM_KIND_MK4>(a.x_vals, a.x_meta, a.x_n, a.x_k, a.x_blocks, a.x_k_steps, a.x_out, b, lane, lut,
                                      tid, nthreads);
            break;
        case NM_KIND_MK5:
            expand_block<NM_KIND_MK5>(a.x_vals, a.x_meta, a.x_n, a.x_k, a.x_blocks, a.x_k_steps, a.x_out, b, lane, lut,
                                      tid, nthreads);
            break;
    }
}

template <int KIND, int WN_, int WM_, int FN_, int FM_, int NST>
struct Geometry {
    using K = Kind<KIND>;
    static constexpr int WN = WN_, WM = WM_, FN = FN_, FM = FM_;
    static constexpr int NW = WN * WM;                               // waves per workgroup (4 or 8)
    static constexpr int BN = WN * FN * 16;
    static constexpr int BM = WM * FM * 16;
    static constexpr int XB = BM * 128;                              // X bytes per slot
    static constexpr int WVB = K::kSp ? (BN / 16) * kVBlock : BN * 128;  // weight value bytes per slot
    static constexpr int WMB = K::kSp ? (BN / 16) * kMBlock : 0;         // weight position bytes per slot
    static constexpr int SLOT = XB + WVB + WMB;
    static constexpr int XI = BM / (8 * NW);                         // X loads per wave per k-step
    static constexpr int WB = (BN / 16) / NW;                        // weight blocks per wave (compact kinds)
    static constexpr int WI = K::kDecode ? WB * K::LOADS                          // weight loads per wave
                              : KIND == NM_KIND_SP42 ? (BN / 16) / NW * 2 : BN / (8 * NW);
    static constexpr int DMA = XI + WI;                              // vector-memory loads per wave per k-step
    static constexpr int CPR = FN * 4;                               // 4-channel chunks per staged row
    static constexpr int RPI = 64 / CPR;                             // staged rows read per instruction
    static constexpr int ROWB = FN * 64 + 16;                        // padded bytes per staged int32 row
    static constexpr int EPI = NW * 16 * ROWB;
    // ring depth: as asked, or as deep as 160 KB of LDS allows
    static constexpr int RING = NST * SLOT <= 160 * 1024 - 4096 ? NST : (160 * 1024 - 4096) / SLOT;
    static constexpr int LDSB = RING * SLOT > EPI ? RING * SLOT : EPI;
    static_assert((NW == 4 || NW == 8) && RING >= 2 && 64 % CPR == 0 && BM % (8 * NW) == 0, "tile shape");
    static_assert(KIND == NM_KIND_DENSE ? BN % (8 * NW) == 0 : (BN / 16) % NW == 0,
                  "weight loads split evenly over the waves");
    static_assert(LDSB + K::LUT * 8 <= 160 * 1024, "LDS budget");
};

// The stages of an output-split tile (WN x WM waves, each FN x FM
// accumulators).
template <class G, int KIND>
struct OutSplit {
    using K = Kind<KIND>;
    static constexpr int BN = G::BN, BM = G::BM, FN = G::FN, FM = G::FM, NW = G::NW;
    static constexpr int WJ = KIND == NM_KIND_SP42 ? (BN / 16) / NW : K::kDecode ? G::WB : BN / (8 * NW);

    // Per-lane byte offsets of one tile's loads at k-step 0: the X row chunks
    // and the weight blocks (or dense weight row chunks).  A k-step adds the
    // same amount to every lane, so each load is a 32-bit offset from a
    // scalar base that advances with the k-step (X and the weights hold fewer
    // than 2^32 bytes, checked on the host).  Rows of X past m, and weight
    // rows past n, read a valid row instead: their outputs are never stored.
    struct Cursor {
        uint32_t x[G::XI];
        uint32_t w[WJ];
        uint32_t m[KIND == NM_KIND_DENSE ? 1 : WJ];
    };

    static __device__ __forceinline__ Cursor cursor(const GemmArgs &a, int wave, int lane, int tok0, int ch0) {
        Cursor c;
#pragma unroll
        for (int j = 0; j < G::XI; ++j) {
            const int r = 8 * (NW * j + wave) + (lane >> 3);
            const int cc = (lane & 7) ^ (r & 7);
            const int tok = tok0 + r < a.m ? tok0 + r : a.m - 1;
            c.x[j] = (uint32_t)tok * (uint32_t)a.k + (uint32_t)cc * 16;
        }
        if constexpr (KIND == NM_KIND_SP42 || K::kDecode) {
            const int f0 = ch0 >> 4;
            constexpr int VB = KIND == NM_KIND_SP42 ? 16 : K::VB, MB = KIND == NM_KIND_SP42 ? 4 : K::MB;
#pragma unroll
            for (int j = 0; j < WJ; ++j) {
                const int bl = NW * j + wave;              // weight block of the slot
                int f = f0 + bl;
                f = f < a.n_frags ? f : a.n_frags - 1;
                const uint32_t b0 = (uint32_t)f * (uint32_t)a.k_steps;
                c.w[j] = (b0 * 64 + lane) * VB;
                c.m[j] = (b0 * 64 + lane) * MB;
            }
        } else {
#pragma unroll
            for (int j = 0; j < WJ; ++j) {
                const int r = 8 * (NW * j + wave) + (lane >> 3);
                const int cc = (lane & 7) ^ (r & 7);
                const int row = ch0 + r < a.n ? ch0 + r : a.n - 1;
                c.w[j] = (uint32_t)row * (uint32_t)a.k + (uint32_t)cc * 16;
            }
        }
        return c;
    }

    // Fill ring slot st with k-step s of the tile of cursor c: the X slice,
    // and for the stored kinds the weight slice.  Past k the packed weight is
    // zero, so X may hold anything there (its loads are clamped to the row);
    // for a dense weight the tail k-step is staged with zeros instead.
    static __device__ __forceinline__ void issue(const GemmArgs &a, const Cursor &c, int8_t *lds, uint32_t lds0,
                                                 int wave, int lane, int s, int st) {
        const uint32_t slot = lds0 + st * G::SLOT;
        if (s * 128 + 128 <= a.k) {
            const int8_t *xb = a.X + (size_t)s * 128;
#pragma unroll
            for (int j = 0; j < G::XI; ++j) dma16o(xb, c.x[j], slot + (NW * j + wave) * 1024);
        } else {
            // last k-step of a k that is not a multiple of 128: clamp to the row
#pragma unroll
            for (int j = 0; j < G::XI; ++j) {
                const int r = 8 * (NW * j + wave) + (lane >> 3);
                const uint32_t cc16 = (uint32_t)(((lane & 7) ^ (r & 7)) * 16);
                const uint32_t kk = (uint32_t)s * 128 + cc16 < (uint32_t)a.k ? (uint32_t)s * 128 + cc16
                                                                              : (uint32_t)a.k - 16;
                dma16o(a.X, c.x[j] - cc16 + kk, slot + (NW * j + wave) * 1024);
            }
        }
        if constexpr (KIND == NM_KIND_SP42) {
            const int8_t *vb = a.A + (size_t)s * kVBlock;
            const uint8_t *mb = a.meta + (size_t)s * kMBlock;
#pragma unroll
            for (int j = 0; j < WJ; ++j) {
                const int bl = NW * j + wave;
                dma16o(vb, c.w[j], slot + G::XB + bl * kVBlock);
                dma4o(mb, c.m[j], slot + G::XB + G::WVB + bl * kMBlock);
            }
        } else if constexpr (KIND == NM_KIND_DENSE) {
            if (s * 128 + 128 <= a.k) {
                const int8_t *wb = a.A + (size_t)s * 128;
#pragma unroll
                for (int j = 0; j < WJ; ++j) dma16o(wb, c.w[j], slot + G::XB + (NW * j + wave) * 1024);
            } else {
                // tail k-step of a dense weight: plain loads, zeros past k
#pragma unroll
                for (int j = 0; j < WJ; ++j) {
                    const int r = 8 * (NW * j + wave) + (lane >> 3);
                    const uint32_t cc16 = (uint32_t)(((lane & 7) ^ (r & 7)) * 16);
                    const uint32_t kk = (uint32_t)s * 128 + cc16;
                    v4i v = v4i{0, 0, 0, 0};
                    if (kk < (uint32_t)a.k) v = *(const v4i *)(a.A + (c.w[j] - cc16 + kk));
                    *(v4i *)(lds + st * G::SLOT + G::XB + (NW * j + wave) * 1024 + lane * 16) = v;
                }
            }
        }
    }

    // Compact kinds: this wave's compact blocks of k-step s into registers.
    static __device__ __forceinline__ void wload_step(const GemmArgs &a, const Cursor &c, int s,
                                                      WRegs<KIND> (&r)[WJ]) {
        if constexpr (K::kDecode) {
            const int8_t *vb = a.A + (size_t)s * 64 * K::VB;
            const uint8_t *mb = a.meta + (size_t)s * 64 * K::MB;
#pragma unroll
            for (int j = 0; j < WJ; ++j) wload<KIND>(r[j], vb + c.w[j], mb + c.m[j]);
        }
    }

    // Compact kinds: expand the registers into the weight area of slot st.
    static __device__ __forceinline__ void expand_step(int8_t *lds, const uint2 *lut, int wave, int lane, int st,
                                                       const WRegs<KIND> (&r)[WJ]) {
        if constexpr (K::kDecode) {
#pragma unroll
            for (int j = 0; j < WJ; ++j)
                expand_to_lds<KIND, G::WVB>(r[j], lut, lds + st * G::SLOT + G::XB, NW * j + wave, lane);
        }
    }

    // One k-step of the wave's FN x FM accumulators from ring slot st.
    static __device__ __forceinline__ void compute(const int8_t *lds, int wn, int wm, int lane, int st,
                                                   v4i (&acc)[FN][FM]) {
        const int lg = lane >> 4;
        const int8_t *xs = lds + st * G::SLOT;
        const int8_t *ws = xs + G::XB;
        if constexpr (K::kSp) {
            v4i av[FN];
            int ai[FN];
#pragma unroll
            for (int i = 0; i < FN; ++i) {
                const int bl = wn * FN + i;
                av[i] = *(const v4i *)(ws + bl * kVBlock + lane * 16);
                ai[i] = *(const int *)(ws + G::WVB + bl * kMBlock + lane * 4);
            }
#pragma unroll
            for (int j = 0; j < FM; ++j) {
                const int r = (wm * FM + j) * 16 + (lane & 15);
                const int8_t *rowp = xs + r * 128;
                const v4i blo = *(const v4i *)(rowp + ((lg ^ (r & 7)) << 4));
                const v4i bhi = *(const v4i *)(rowp + (((lg + 4) ^ (r & 7)) << 4));
                const v8i b = {blo[0], blo[1], blo[2], blo[3], bhi[0], bhi[1], bhi[2], bhi[3]};
#pragma unroll
                for (int i = 0; i < FN; ++i)
                    acc[i][j] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(av[i], b, acc[i][j], ai[i], 0, 0);
            }
        } else {
            v4i alo[FN], ahi[FN];
#pragma unroll
            for (int i = 0; i < FN; ++i) {
                const int r = (wn * FN + i) * 16 + (lane & 15);
                const int8_t *rowp = ws + r * 128;
                alo[i] = *(const v4i *)(rowp + ((lg ^ (r & 7)) << 4));
                ahi[i] = *(const v4i *)(rowp + (((lg + 4) ^ (r & 7)) << 4));
            }
#pragma unroll
            for (int j = 0; j < FM; ++j) {
                const int r = (wm * FM + j) * 16 + (lane & 15);
                const int8_t *rowp = xs + r * 128;
                const v4i blo = *(const v4i *)(rowp + ((lg ^ (r & 7)) << 4));
                const v4i bhi = *(const v4i *)(rowp + (((lg + 4) ^ (r & 7)) << 4));
#pragma unroll
                for (int i = 0; i < FN; ++i) {
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(alo[i], blo, acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ahi[i], bhi, acc[i][j], 0, 0, 0);
                }
            }
        }
    }

    // Epilogue of the wave's part of a tile through its private staging area
    // stg (16 rows of ROWB bytes): 16 tokens at a time, the FN accumulators
    // become int32 rows, read back row-contiguously, so that every store
    // instruction writes whole rows of the wave's tile.  With split_k > 1 the
    // rows go to the partial-sum workspace instead.
    static __device__ __forceinline__ void store(const GemmArgs &a, int8_t *stg, int lane, int wn, int wm, int tok0,
                                                 int ch0, int split, const v4i (&acc)[FN][FM]) {
        const int lg = lane >> 4;
        const int ec = lane % G::CPR;                     // 4-channel chunk this lane stores
        const int er = lane / G::CPR;                     // row offset within a read group
        const int ch = ch0 + wn * FN * 16 + ec * 4;       // first of the lane's 4 channels
        const bool ch_ok = ch < a.n;
        const EpiScale sc = load_scale(a, ch);
        const __amdgpu_buffer_rsrc_t prsrc = partial_rsrc(a);
        constexpr int NR = 16 / G::RPI;                   // staged rows each lane stores per 16 tokens
#pragma unroll
        for (int j = 0; j < FM; ++j) {
#pragma unroll
            for (int i = 0; i < FN; ++i)
                *(v4i *)(stg + (lane & 15) * G::ROWB + (i * 16 + 4 * lg) * 4) = acc[i][j];
            // all reads first, then the stores: one wait for the reads, none between stores
            v4i v[NR];
#pragma unroll
            for (int r = 0; r < NR; ++r) v[r] = *(const v4i *)(stg + (r * G::RPI + er) * G::ROWB + ec * 16);
#pragma unroll
            for (int r = 0; r < NR; ++r) {
                const int tok = tok0 + (wm * FM + j) * 16 + r * G::RPI + er;
                if (tok < a.m && ch_ok) {
                    if (a.split_k == 1)
                        emit_out(a, tok, ch, v[r], sc);
                    else
                        publish_partial(a, prsrc, split, tok, ch, v[r]);
                }
            }
        }
    }
};

template <int KIND, int WN, int WM, int FN, int FM, int NST>
__global__ __launch_bounds__(64 * WN * WM) void k_gemm(GemmArgs a) {
    using G = Geometry<KIND, WN, WM, FN, FM, NST>;
    using O = OutSplit<G, KIND>;
    using K = Kind<KIND>;
    constexpr int BN = G::BN, BM = G::BM;
    constexpr int R = G::RING;

    __shared__ __attribute__((aligned(1024))) int8_t lds[G::LDSB];
    __shared__ uint2 lut[K::LUT];
    __shared__ int s_last;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) int8_t *)lds;
    static_assert(G::LDSB >= 256 * 8, "room for the expansion table of a tail workgroup");
    if ((int)blockIdx.x >= a.gemm_grid) {
        expand_tail(a, (uint2 *)lds);
        return;
    }

    const int lid = map_block(blockIdx.x, (int)gridDim.x < a.gemm_grid ? (int)gridDim.x : a.gemm_grid);
    int tn, rest;
    tile_order(lid, a.tiles_n, a.tiles_m * a.split_k, a.group_rows, &tn, &rest);
    const int split = rest % a.split_k;
    const int tm = rest / a.split_k;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wn = wave % WN, wm = wave / WN;
    const int tok0 = tm * BM;
    const int ch0 = tn * BN;
    const int s_begin = (int)((int64_t)split * a.k_steps / a.split_k);
    const int s_end = (int)((int64_t)(split + 1) * a.k_steps / a.split_k);
    const int nsteps = s_end - s_begin;

    v4i acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = v4i{0, 0, 0, 0};

    const typename O::Cursor cur = O::cursor(a, wave, lane, tok0, ch0);
    WRegs<KIND> wr[O::WJ];
#pragma unroll
    for (int i = 0; i < R - 1; ++i)
        if (i < nsteps) O::issue(a, cur, lds, lds0, wave, lane, s_begin + i, i);
    if constexpr (K::kDecode) {
        // the compact weights of the first R - 1 k-steps, expanded in order,
        // and the next k-step's loaded into registers; the lookup table is
        // built while the first loads are in flight
        if (nsteps > 0) O::wload_step(a, cur, s_begin, wr);
        fill_lut<KIND>(lut, tid, 64 * WN * WM);
        __syncthreads();
#pragma unroll
        for (int i = 0; i < R - 1; ++i)
            if (i < nsteps) {
                O::expand_step(lds, lut, wave, lane, i, wr);
                if (i + 1 < nsteps) O::wload_step(a, cur, s_begin + i + 1, wr);
            }
    }
    for (int it = 0; it < nsteps; ++it) {
        // k-step it was issued NST-1 iterations ago; only the loads of later
        // k-steps may remain in flight.  The barrier then publishes every
        // wave's slot (X and expanded weights) and frees the slot computed in
        // the previous iteration.
        const int later = nsteps - 1 - it < R - 2 ? nsteps - 1 - it : R - 2;
        wait_later_then_barrier<R - 2, G::DMA>(later);
        const int nx = it + R - 1;
        if (nx < nsteps) {
            if constexpr (K::kDecode) {
                O::expand_step(lds, lut, wave, lane, nx % R, wr);      // k-step nx, loaded one iteration ago
                O::issue(a, cur, lds, lds0, wave, lane, s_begin + nx, nx % R);
                if (nx + 1 < nsteps) O::wload_step(a, cur, s_begin + nx + 1, wr);
            } else {
                O::issue(a, cur, lds, lds0, wave, lane, s_begin + nx, nx % R);
            }
        }
        O::compute(lds, wn, wm, lane, it % R, acc);
    }

    __syncthreads();  // every wave is done with the ring
    O::store(a, lds + wave * 16 * G::ROWB, lane, wn, wm, tok0, ch0, split, acc);
    if (a.split_k == 1) return;

    // Split-K: the last split to arrive adds every partial (integer addition:
    // any order gives the same result) and writes the outputs.
    if (!arrive_last(a, tm * a.tiles_n + tn, &s_last)) return;
    const int ec = lane % G::CPR, er = lane / G::CPR;
    const int ch = ch0 + wn * FN * 16 + ec * 4;
    const bool ch_ok = ch < a.n;
    const EpiScale sc = load_scale(a, ch);
    const __amdgpu_buffer_rsrc_t prsrc = partial_rsrc(a);
#pragma unroll
    for (int j = 0; j < FM; ++j)
#pragma unroll
        for (int r0 = 0; r0 < 16; r0 += G::RPI) {
            const int tok = tok0 + (wm * FM + j) * 16 + r0 + er;
            if (tok < a.m && ch_ok) emit_out(a, tok, ch, merge_partials(a, prsrc, tok, ch), sc);
        }
}

// ---------------------------------------------------------------------------
// k-sliced variant for shapes with few output tiles (small token counts).
// Each of the 4 waves computes the whole tile_n x tile_m tile over its own
// quarter of the k-steps (k-step s goes to wave s % 4), through a ring of
// LDS slots that only it fills and reads: no workgroup barrier in the main
// loop, and FN x FM matrix instructions per wave per k-step to cover the LDS
// latency.  The four partial tiles are added through LDS at the end -- a
// split of the reduction merged in the final stage without leaving the CU.

template <int KIND, int FN, int FM, int NST>
struct GeometryKS {
    using K = Kind<KIND>;
    // 1:4, 1:8 and 2:8: the compact bytes reach the ring by direct-to-LDS
    // loads like X (RAWV value bytes and RAWM position bytes per k-step, the
    // positions padded to 4 bytes per lane), and the compute stage expands
    // them into the 4:2 operand in registers (no expanded copy in LDS)
    static constexpr bool kRaw = K::kDecode && K::kSp;
    static constexpr int BN = FN * 16;
    static constexpr int BM = FM * 16;
    static constexpr int XB = BM * 128;
    static constexpr int WVB = kRaw ? 0 : K::kSp ? (BN / 16) * kVBlock : BN * 128;
    static constexpr int WMB = kRaw ? 0 : K::kSp ? (BN / 16) * kMBlock : 0;
    static constexpr int RAWV = kRaw ? FN * 64 * K::VB : 0;
    static constexpr int RAWM = kRaw ? FN * 256 : 0;
    static constexpr int SLOT = XB + WVB + WMB + RAWV + RAWM;
    static constexpr int XI = BM / 8;                                  // X loads per k-step (one wave)
    static constexpr int WI = kRaw ? FN * (K::VB / 4 + 1)
                              : K::kDecode ? FN * K::LOADS : KIND == NM_KIND_SP42 ? FN * 2 : BN / 8;
    static constexpr int DMA = XI + WI;
    static constexpr int RING = 4 * NST * SLOT <= 160 * 1024 - 4096 ? NST : (160 * 1024 - 4096) / (4 * SLOT);
    static constexpr int ROWB = BN * 4 + 16;                           // padded staged row (int32)
    static constexpr int RED = 4 * BM * ROWB;
    static constexpr int LDSB = 4 * RING * SLOT > RED ? 4 * RING * SLOT : RED;
    static constexpr int CPR = BN / 4;                                 // 16-byte chunks per output row
    static_assert(RING >= 2 && BM % 8 == 0 && BN % 16 == 0, "tile shape");
};

template <int KIND, int FN, int FM, int NST>
__global__ __launch_bounds__(256) void k_gemm_ks(GemmArgs a) {
    using G = GeometryKS<KIND, FN, FM, NST>;
    using K = Kind<KIND>;
    constexpr int BN = G::BN, BM = G::BM, R = G::RING;

    __shared__ __attribute__((aligned(1024))) int8_t lds[G::LDSB];
    __shared__ uint2 lut[K::LUT];
    __shared__ int s_last;
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) int8_t *)lds;
    static_assert(G::LDSB >= 256 * 8, "room for the expansion table of a tail workgroup");
    if ((int)blockIdx.x >= a.gemm_grid) {
        expand_tail(a, (uint2 *)lds);
        return;
    }

    const int lid = map_block(blockIdx.x, (int)gridDim.x < a.gemm_grid ? (int)gridDim.x : a.gemm_grid);
    const int tn = lid % a.tiles_n;
    const int rest = lid / a.tiles_n;
    const int split = rest % a.split_k;
    const int tm = rest / a.split_k;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lg = lane >> 4;
    const int tok0 = tm * BM;
    const int ch0 = tn * BN;
    const int s_begin = (int)((int64_t)split * a.k_steps / a.split_k);
    const int s_end = (int)((int64_t)(split + 1) * a.k_steps / a.split_k);
    const int nsteps = s_end - s_begin > wave ? (s_end - s_begin - wave + 3) / 4 : 0;  // this wave's k-steps
    const int f0 = ch0 >> 4;
    const uint32_t ring = lds0 + wave * R * G::SLOT;
    int8_t *ringp = lds + wave * R * G::SLOT;

    v4i acc[FN][FM];
#pragma unroll
    for (int i = 0; i < FN; ++i)
#pragma unroll
        for (int j = 0; j < FM; ++j) acc[i][j] = v4i{0, 0, 0, 0};

    // k-step s into slot st of this wave's ring (same clamping rules as above):
    // X, and the stored weight kinds
    auto issue = [&](int s, int st) {
        const uint32_t slot = ring + st * G::SLOT;
#pragma unroll
        for (int j = 0; j < BM / 8; ++j) {
            const int r = 8 * j + (lane >> 3);
            const int c = (lane & 7) ^ (r & 7);
            const int tok = tok0 + r < a.m ? tok0 + r : a.m - 1;
            const int kk = s * 128 + c * 16 < a.k ? s * 128 + c * 16 : a.k - 16;
            dma16(a.X + (size_t)tok * a.k + kk, slot + j * 1024);
        }
        if constexpr (KIND == NM_KIND_SP42) {
#pragma unroll
            for (int bl = 0; bl < BN / 16; ++bl) {
                int f = f0 + bl;
                f = f < a.n_frags ? f : a.n_frags - 1;
                const size_t b = (size_t)f * a.k_steps + s;
                dma16(a.A + b * kVBlock + lane * 16, slot + G::XB + bl * kVBlock);
                dma4(a.meta + b * kMBlock + lane * 4, slot + G::XB + G::WVB + bl * kMBlock);
            }
        } else if constexpr (KIND == NM_KIND_DENSE) {
#pragma unroll
            for (int j = 0; j < BN / 8; ++j) {
                const int r = 8 * j + (lane >> 3);
                const int c = (lane & 7) ^ (r & 7);
                const int row = ch0 + r < a.n ? ch0 + r : a.n - 1;
                const int kk = s * 128 + c * 16;
                if (s * 128 + 128 <= a.k) {
                    dma16(a.A + (size_t)row * a.k + kk, slot + G::XB + j * 1024);
                } else {  // tail k-step of a dense weight: zeros past k
                    v4i v = v4i{0, 0, 0, 0};
                    if (kk < a.k) v = *(const v4i *)(a.A + (size_t)row * a.k + kk);
                    *(v4i *)(ringp + st * G::SLOT + G::XB + j * 1024 + lane * 16) = v;
                }
            }
        } else if constexpr (G::kRaw) {
            // the FN compact blocks as stored: value bytes as whole dwords
            // (dword i of a block by lane i % 64 of load i / 64), positions one
            // dword per lane (2-byte positions: lanes 32-63 repeat lanes 0-31,
            // landing in the unused half of the 256-byte area)
            constexpr int VB = K::VB, MB = K::MB;
#pragma unroll
            for (int bl = 0; bl < FN; ++bl) {
                int f = f0 + bl;
                f = f < a.n_frags ? f : a.n_frags - 1;
                const size_t b = (size_t)f * a.k_steps + s;
                const int8_t *vb = a.A + b * 64 * VB;
#pragma unroll
                for (int i = 0; i < VB / 4; ++i)
                    dma4(vb + (i * 64 + lane) * 4, slot + G::XB + G::WVB + G::WMB + bl * 64 * VB + i * 256);
                const uint8_t *mb = a.meta + b * 64 * MB;
                dma4(mb + (MB == 4 ? lane : (lane & 31)) * 4, slot + G::XB + G::WVB + G::WMB + G::RAWV + bl * 256);
            }
        }
    };
    // mask layouts (3:8-5:8; the loop below calls these only for them): the
    // FN blocks of k-step s into registers, and their expansion into dense
    // rows of slot st
    WRegs<KIND> wr[FN];
    auto wload_step = [&](int s) {
        if constexpr (K::kDecode) {
#pragma unroll
            for (int bl = 0; bl < FN; ++bl) {
                int f = f0 + bl;
                f = f < a.n_frags ? f : a.n_frags - 1;
                const size_t b = (size_t)f * a.k_steps + s;
                wload<KIND>(wr[bl], a.A + (b * 64 + lane) * K::VB, a.meta + (b * 64 + lane) * K::MB);
            }
        }
    };
    auto expand_step = [&](int st) {
        if constexpr (K::kDecode) {
#pragma unroll
            for (int bl = 0; bl < FN; ++bl) expand_to_lds<KIND, G::WVB>(wr[bl], lut, ringp + st * G::SLOT + G::XB, bl, lane);
        }
    };
    // 1:4, 1:8, 2:8: block bl of slot st's compact bytes, read from the ring
    // and expanded into this lane's 4:2 operand (values and position word)
    auto raw_operand = [&](int st, int bl, v4i &av, int &ai) {
        if constexpr (G::kRaw) {
            constexpr int VB = K::VB, MB = K::MB;
            const int8_t *raw = ringp + st * G::SLOT + G::XB;
            WRegs<KIND> r;
            const int8_t *v = raw + bl * 64 * VB + lane * VB;
            if constexpr (VB == 8) {
                const v2u t = *(const v2u *)v;
                r.v[0] = t[0];
                r.v[1] = t[1];
            } else {
                static_assert(VB == 4, "compact 4:2 value bytes per lane");
                r.v[0] = *(const uint32_t *)v;
            }
            const int8_t *m = raw + G::RAWV + bl * 256 + lane * MB;
            r.m = MB == 4 ? *(const uint32_t *)m : (uint32_t) * (const uint16_t *)m;
            uint32_t idx;
            expand_sp42<KIND>(r, lut, av, idx);
            ai = (int)idx;
        }
    };
    auto compute = [&](int st) {
        const int8_t *xs = ringp + st * G::SLOT;
        const int8_t *ws = xs + G::XB;
        if constexpr (K::kSp) {
            v4i av[FN];
            int ai[FN];
#pragma unroll
            for (int i = 0; i < FN; ++i) {
                if constexpr (G::kRaw) {
                    raw_operand(st, i, av[i], ai[i]);
                } else {
                    av[i] = *(const v4i *)(ws + i * kVBlock + lane * 16);
                    ai[i] = *(const int *)(ws + G::WVB + i * kMBlock + lane * 4);
                }
            }
#pragma unroll
            for (int j = 0; j < FM; ++j) {
                const int r = j * 16 + (lane & 15);
                const int8_t *rowp = xs + r * 128;
                const v4i blo = *(const v4i *)(rowp + ((lg ^ (r & 7)) << 4));
                const v4i bhi = *(const v4i *)(rowp + (((lg + 4) ^ (r & 7)) << 4));
                const v8i b = {blo[0], blo[1], blo[2], blo[3], bhi[0], bhi[1], bhi[2], bhi[3]};
#pragma unroll
                for (int i = 0; i < FN; ++i)
                    acc[i][j] = __builtin_amdgcn_smfmac_i32_16x16x128_i8(av[i], b, acc[i][j], ai[i], 0, 0);
            }
        } else {
            v4i alo[FN], ahi[FN];
#pragma unroll
            for (int i = 0; i < FN; ++i) {
                const int r = i * 16 + (lane & 15);
                const int8_t *rowp = ws + r * 128;
                alo[i] = *(const v4i *)(rowp + ((lg ^ (r & 7)) << 4));
                ahi[i] = *(const v4i *)(rowp + (((lg + 4) ^ (r & 7)) << 4));
            }
#pragma unroll
            for (int j = 0; j < FM; ++j) {
                const int r = j * 16 + (lane & 15);
                const int8_t *rowp = xs + r * 128;
                const v4i blo = *(const v4i *)(rowp + ((lg ^ (r & 7)) << 4));
                const v4i bhi = *(const v4i *)(rowp + (((lg + 4) ^ (r & 7)) << 4));
#pragma unroll
                for (int i = 0; i < FN; ++i) {
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(alo[i], blo, acc[i][j], 0, 0, 0);
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(ahi[i], bhi, acc[i][j], 0, 0, 0);
                }
            }
        }
    };

    // k-step t of this wave is s_begin + wave + 4 t
#pragma unroll
    for (int i = 0; i < R - 1; ++i)
        if (i < nsteps) issue(s_begin + wave + 4 * i, i);
    if constexpr (G::kRaw) {
        fill_lut<KIND>(lut, tid, 256);
        __syncthreads();
    } else if constexpr (K::kDecode) {
        // the lookup table is built while the first loads are in flight
        if (nsteps > 0) wload_step(s_begin + wave);
        fill_lut<KIND>(lut, tid, 256);
        __syncthreads();
#pragma unroll
        for (int i = 0; i < R - 1; ++i)
            if (i < nsteps) {
                expand_step(i);
                if (i + 1 < nsteps) wload_step(s_begin + wave + 4 * (i + 1));
            }
    }
    for (int t = 0; t < nsteps; ++t) {
        const int later = nsteps - 1 - t < R - 2 ? nsteps - 1 - t : R - 2;
        wait_later<R - 2, G::DMA>(later);  // this wave's slot t is in LDS, its reads of slot t-1 done
        const int nx = t + R - 1;
        if (nx < nsteps) {
            if constexpr (K::kDecode && !G::kRaw) {
                expand_step(nx % R);
                issue(s_begin + wave + 4 * nx, nx % R);
                if (nx + 1 < nsteps) wload_step(s_begin + wave + 4 * (nx + 1));
            } else {
                issue(s_begin + wave + 4 * nx, nx % R);
            }
        }
        compute(t % R);
    }

    // Add the four waves' partial tiles through LDS, then write rows.
    __syncthreads();  // every wave is done with its ring
    int8_t *stg = lds + wave * BM * G::ROWB;
#pragma unroll
    for (int j = 0; j < FM; ++j)
#pragma unroll
        for (int i = 0; i < FN; ++i)
            *(v4i *)(stg + (j * 16 + (lane & 15)) * G::ROWB + (i * 16 + 4 * lg) * 4) = acc[i][j];
    __syncthreads();
    const __amdgpu_buffer_rsrc_t prsrc = partial_rsrc(a);
    constexpr int CHUNKS = BM * G::CPR;
    static_assert(256 % G::CPR == 0, "a thread keeps its channel chunk across rows");
    const int cc = tid % G::CPR, ch = ch0 + cc * 4;   // the same for every row this thread stores
    const EpiScale sc = load_scale(a, ch);
    for (int c = tid; c < CHUNKS; c += 256) {
        const int row = c / G::CPR;
        const int tok = tok0 + row;
        v4i v = v4i{0, 0, 0, 0};
#pragma unroll
        for (int w = 0; w < 4; ++w) v += *(const v4i *)(lds + w * BM * G::ROWB + row * G::ROWB + cc * 16);
        if (tok < a.m && ch < a.n) {
            if (a.split_k == 1)
                emit_out(a, tok, ch, v, sc);
            else
                publish_partial(a, prsrc, split, tok, ch, v);
        }
    }
    if (a.split_k == 1) return;
    if (!arrive_last(a, tm * a.tiles_n + tn, &s_last)) return;
    for (int c = tid; c < CHUNKS; c += 256) {
        const int tok = tok0 + c / G::CPR;
        if (tok < a.m && ch < a.n) emit_out(a, tok, ch, merge_partials(a, prsrc, tok, ch), sc);
    }
}

// ---------------------------------------------------------------------------
// Expansion of a compact weight once per call (plan.expand = 1): one thread
// per lane of every (fragment, k-step) block, the same expansion as inside the
// GEMM kernels, written out as the 4:2 operand blocks of the SP42 layout
// (C14, C18, C28) or as dense W [n x k] row-major (mask layouts; rows >= n and
// columns >= k of the padded blocks are not written).  4 blocks per
// workgroup; blocks = n_frags * k_steps.
// One wave expands block b of a compact weight (1:4, 1:8, 2:8 to the 4:2
// operand; 3:8-5:8 to dense rows of W) into out.  The workgroup's lookup
// table is built while the block's bytes are in flight; every wave of the
// workgroup must call this (it holds a barrier), waves past the last block
// load a valid block and store nothing.
template <int KIND>
__device__ __forceinline__ void expand_block(const int8_t *__restrict__ vals, const uint8_t *__restrict__ meta, int n,
                                             int k, int blocks, int k_steps, int8_t *out, int b, int lane, uint2 *lut,
                                             int tid, int nthreads) {
    WRegs<KIND> r;
    const int64_t o = (int64_t)(b < blocks ? b : blocks - 1) * 64 + lane;
    wload<KIND>(r, vals + o * Kind<KIND>::VB, meta + o * Kind<KIND>::MB);
    fill_lut<KIND>(lut, tid, nthreads);
    __syncthreads();
    if (b >= blocks) return;
    if constexpr (Kind<KIND>::kSp) {
        v4i v;
        uint32_t idx;
        expand_sp42<KIND>(r, lut, v, idx);
        *(v4i *)(out + o * 16) = v;
        *(uint32_t *)(out + (int64_t)blocks * kVBlock + o * 4) = idx;
    } else {
        v4i c0, c1;
        expand_dense<KIND>(r, lut, c0, c1);
        const int f = b / k_steps, s = b - f * k_steps;
        const int row = f * kFragRows + (lane & 15);
        const int col = s * kKStep + 32 * (lane >> 4);
        if (row < n) {
            int8_t *dst = out + (int64_t)row * k + col;
            if (col < k) *(v4i *)dst = c0;          // k is a multiple of 16: a chunk is wholly in or out
            if (col + 16 < k) *(v4i *)(dst + 16) = c1;
        }
    }
}

template <int KIND>
__global__ __launch_bounds__(256) void k_expand(const int8_t *__restrict__ vals, const uint8_t *__restrict__ meta,
                                               int n, int k, int blocks, int k_steps, int8_t *out) {
    __shared__ uint2 lut[Kind<KIND>::LUT];
    expand_block<KIND>(vals, meta, n, k, blocks, k_steps, out, blockIdx.x * 4 + (threadIdx.x >> 6), threadIdx.x & 63,
                       lut, threadIdx.x, 256);
}

__global__ void k_zero(int *p, size_t n4, unsigned char *tail, int tail_bytes) {
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) p[i] = 0;
    if (blockIdx.x == 0 && (int)threadIdx.x < tail_bytes) tail[threadIdx.x] = 0;
}

template <int KIND, int T>
int launch_one(const GemmArgs &args, int grid, void *stream) {
    constexpr TileCfg t = kTiles[T];
    if constexpr (t.layout == kKSliced)
        hipLaunchKernelGGL((k_gemm_ks<KIND, t.fn, t.fm, t.nst>), dim3(grid), dim3(kThreads), 0,
                           (hipStream_t)stream, args);
    else
        hipLaunchKernelGGL((k_gemm<KIND, t.wn, t.wm, t.fn, t.fm, t.nst>), dim3(grid), dim3(64 * t.wn * t.wm), 0,
                           (hipStream_t)stream, args);
    return (int)hipGetLastError();
}

template <int KIND, int T = 0>
int launch_kind(int tile, const GemmArgs &args, int grid, void *stream) {
    if constexpr (T < kNumTiles) {
        if (tile == T) return launch_one<KIND, T>(args, grid, stream);
        return launch_kind<KIND, T + 1>(tile, args, grid, stream);
    }
    return (int)hipErrorInvalidValue;
}

}  // namespace

template <int KIND>
int launch_expand_kind(const int8_t *vals, const uint8_t *meta, int n, int k, int8_t *out, void *stream) {
    const int blocks = ((n + kFragRows - 1) / kFragRows) * ((k + kKStep - 1) / kKStep);
    hipLaunchKernelGGL(k_expand<KIND>, dim3((blocks + 3) / 4), dim3(256), 0, (hipStream_t)stream, vals, meta, n, k,
                       blocks, (k + kKStep - 1) / kKStep, out);
    return (int)hipGetLastError();
}

int launch_expand(int kind, const int8_t *vals, const uint8_t *meta, int n, int k, int8_t *out, void *stream) {
    switch (kind) {
        case NM_KIND_C14: return launch_expand_kind<NM_KIND_C14>(vals, meta, n, k, out, stream);
        case NM_KIND_C18: return launch_expand_kind<NM_KIND_C18>(vals, meta, n, k, out, stream);
        case NM_KIND_C28: return launch_expand_kind<NM_KIND_C28>(vals, meta, n, k, out, stream);
        case NM_KIND_MK3: return launch_expand_kind<NM_KIND_MK3>(vals, meta, n, k, out, stream);
        case NM_KIND_MK4: return launch_expand_kind<NM_KIND_MK4>(vals, meta, n, k, out, stream);
        case NM_KIND_MK5: return launch_expand_kind<NM_KIND_MK5>(vals, meta, n, k, out, stream);
    }
    return (int)hipErrorInvalidValue;
}

int launch_gemm(int kind, int tile, const GemmArgs &args, int grid, void *stream) {
    switch (kind) {
        case NM_KIND_SP42: return launch_kind<NM_KIND_SP42>(tile, args, grid, stream);
        case NM_KIND_C14: return launch_kind<NM_KIND_C14>(tile, args, grid, stream);
        case NM_KIND_DENSE: return launch_kind<NM_KIND_DENSE>(tile, args, grid, stream);
        case NM_KIND_C18: return launch_kind<NM_KIND_C18>(tile, args, grid, stream);
        case NM_KIND_C28: return launch_kind<NM_KIND_C28>(tile, args, grid, stream);
        case NM_KIND_MK3: return launch_kind<NM_KIND_MK3>(tile, args, grid, stream);
        case NM_KIND_MK4: return launch_kind<NM_KIND_MK4>(tile, args, grid, stream);
        case NM_KIND_MK5: return launch_kind<NM_KIND_MK5>(tile, args, grid, stream);
    }
    return (int)hipErrorInvalidValue;
}

typedef _Float16 v8h __attribute__((ext_vector_type(8)));

// Activation quantisation: xq[c] = q8(fp32(x[c]) * inv_scale).  Each thread
// turns 16 binary16 values (two 16-byte loads) into one 16-byte store; the
// count % 16 tail is done one element per thread by block 0.
__global__ __launch_bounds__(256) void k_quantize_f16(const uint16_t *__restrict__ x, size_t chunks,
                                                      float inv_scale, int8_t *__restrict__ xq, int tail) {
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < chunks; i += stride) {
        const v4i lo = *(const v4i *)(x + 16 * i);
        const v4i hi = *(const v4i *)(x + 16 * i + 8);
        const v8h hl = __builtin_bit_cast(v8h, lo), hh = __builtin_bit_cast(v8h, hi);
        v4i out;
#pragma unroll
        for (int w = 0; w < 4; ++w) {
            uint32_t packed = 0;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int idx = 4 * w + e;
                const float v = (float)(idx < 8 ? hl[idx & 7] : hh[idx & 7]) * inv_scale;
                packed |= (uint32_t)(q8(v) & 0xFF) << (8 * e);
            }
            out[w] = (int)packed;
        }
        *(v4i *)(xq + 16 * i) = out;
    }
    if (blockIdx.x == 0 && (int)threadIdx.x < tail) {
        const size_t c = 16 * chunks + threadIdx.x;
        const float v = (float)__builtin_bit_cast(_Float16, x[c]) * inv_scale;
        xq[c] = (int8_t)q8(v);
    }
}

int launch_quantize_f16(const uint16_t *x, int64_t count, float inv_scale, int8_t *xq, void *stream) {
    const size_t chunks = (size_t)count / 16;
    const int tail = (int)(count % 16);
    size_t blocks = (chunks + 255) / 256;
    if (blocks > 8192) blocks = 8192;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_quantize_f16, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, x, chunks,
                       inv_scale, xq, tail);
    return (int)hipGetLastError();
}

int launch_zero(void *ptr, size_t bytes, void *stream) {
    const size_t n4 = bytes / 4;
    const int tail = (int)(bytes % 4);
    size_t blocks = (n4 + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    if (blocks < 1) blocks = 1;
    hipLaunchKernelGGL(k_zero, dim3((unsigned)blocks), dim3(256), 0, (hipStream_t)stream, (int *)ptr, n4,
                       (unsigned char *)ptr + n4 * 4, tail);
    return (int)hipGetLastError();
}

}  // namespace nmspmm
