// Device-side building blocks for the gfx950 GDN kernels: storage traits,
// bf16 rounding, and the 16x16 MFMA tile conventions every kernel shares.
//
// Tile conventions (one 64-lane wavefront, lane l = 16 * lg + li with
// li = l % 16 and lg = l / 16):
//   * an output / accumulator tile D (16 x 16, fp32) lives as 4 floats per
//     lane: lane (li, lg) holds D[4 lg + q][li] for q = 0..3;
//   * a contraction is cut into blocks of 32 along k.  Inside a block a lane
//     supplies the 8 consecutive k = 8 lg + q' (q' = 0..7): an A operand is
//     read as A[row = li][8 lg .. 8 lg + 7], a B operand as B[8 lg ..][col = li],
//     one 16-byte load each for bf16.  A and B use the same k labelling, so
//     the product does not depend on how the hardware orders k inside the
//     instruction;
//   * "P32 order": two accumulator tiles a = 0, 1 whose tile row i stands for
//     row p32_row(a, i) = 8 (i / 4) + 4 a + i % 4 of a 32-row block.  Lane
//     (li, lg) then holds block rows 8 lg .. 8 lg + 7 across the two tiles,
//     which is exactly a B operand over that block: results chain from one
//     MFMA into the next without a trip through LDS.  A tile is produced in
//     P32 order by giving lane li the A-operand row p32_row(a, li).
// bf16 storage uses v_mfma_f32_16x16x32_bf16 (one instruction per block);
// fp32 storage uses eight v_mfma_f32_16x16x4_f32 per block (exact products).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gdn {

constexpr int kChunk = 64;  // tokens per chunk (one wavefront of lanes)
constexpr float kLogAlphaMin = -87.3f;  // ~ log(FLT_MIN): alpha below this acts as 1.2e-38

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two fp32 -> two bf16 packed in one word (low half = lo), round to nearest
// even, by the gfx950 v_cvt_pk_bf16_f32 instruction.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// Row of a 32-row block that tile a (0/1), tile row i stands for (P32 order).
__device__ __forceinline__ int p32_row(int a, int i) { return 8 * (i >> 2) + 4 * a + (i & 3); }

template <class E> struct Tr;

// bf16 storage (uint16_t bit patterns).
template <> struct Tr<uint16_t> {
    using quad = u32x2;  // 4 bf16
    using frag = u32x4;  // 8 bf16
    static __device__ __forceinline__ quad load(const uint16_t *p) { return *(const quad *)p; }
    static __device__ __forceinline__ void store(uint16_t *p, quad v) { *(quad *)p = v; }
    static __device__ __forceinline__ frag load8(const uint16_t *p) { return *(const frag *)p; }
    static __device__ __forceinline__ void store8(uint16_t *p, frag v) { *(frag *)p = v; }
    static __device__ __forceinline__ quad zero() { return quad{0u, 0u}; }
    static __device__ __forceinline__ quad from_f32(f32x4 x) {
        return quad{pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3])};
    }
    static __device__ __forceinline__ f32x4 to_f32(quad v) {
        return f32x4{__uint_as_float(v[0] << 16), __uint_as_float(v[0] & 0xffff0000u),
                     __uint_as_float(v[1] << 16), __uint_as_float(v[1] & 0xffff0000u)};
    }
    static __device__ __forceinline__ frag cat(quad lo, quad hi) {
        return frag{lo[0], lo[1], hi[0], hi[1]};
    }
    static __device__ __forceinline__ quad lo(frag f) { return quad{f[0], f[1]}; }
    // all bits kept (m = ~0) or the quad zeroed (m = 0)
    static __device__ __forceinline__ quad mask(quad v, uint32_t m) { return quad{v[0] & m, v[1] & m}; }
    static __device__ __forceinline__ quad hi(frag f) { return quad{f[2], f[3]}; }
    static __device__ __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                        __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
    }
};

// fp32 storage.
template <> struct Tr<float> {
    using quad = f32x4;
    using frag = f32x8;
    static __device__ __forceinline__ quad load(const float *p) { return *(const quad *)p; }
    static __device__ __forceinline__ void store(float *p, quad v) { *(quad *)p = v; }
    static __device__ __forceinline__ frag load8(const float *p) { return cat(load(p), load(p + 4)); }
    static __device__ __forceinline__ void store8(float *p, frag v) {
        store(p, quad{v[0], v[1], v[2], v[3]});
        store(p + 4, quad{v[4], v[5], v[6], v[7]});
    }
    static __device__ __forceinline__ quad zero() { return quad{0.f, 0.f, 0.f, 0.f}; }
    static __device__ __forceinline__ quad from_f32(f32x4 x) { return x; }
    static __device__ __forceinline__ f32x4 to_f32(quad v) { return v; }
    static __device__ __forceinline__ frag cat(quad lo, quad hi) {
        return frag{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    }
    static __device__ __forceinline__ quad lo(frag f) { return quad{f[0], f[1], f[2], f[3]}; }
    static __device__ __forceinline__ quad mask(quad v, uint32_t m) {
        return quad{__uint_as_float(__float_as_uint(v[0]) & m), __uint_as_float(__float_as_uint(v[1]) & m),
                    __uint_as_float(__float_as_uint(v[2]) & m), __uint_as_float(__float_as_uint(v[3]) & m)};
    }
    static __device__ __forceinline__ quad hi(frag f) { return quad{f[4], f[5], f[6], f[7]}; }
    static __device__ __forceinline__ f32x4 mma(frag a, frag b, f32x4 c) {
#pragma unroll
        for (int s = 0; s < 8; ++s) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], b[s], c, 0, 0, 0);
        return c;
    }
};

// Operand of one 32-wide k block read from a row of memory (LDS or global):
// k = base + 8 lg + q', q' = 0..7.
template <class E>
__device__ __forceinline__ typename Tr<E>::frag load_frag(const E *row_base, int lg) {
    return Tr<E>::load8(row_base + 8 * lg);
}

// Operand fragment whose k index runs down the rows of a row-major LDS tile
// M (row stride ld elements): lane (li, lg) receives M[row0 + 8 lg + q'][col]
// for q' = 0..7, with col = colbase + li, or, for tile a of a P32 pair,
// col = colbase + p32_row(a, li).  bf16 uses the gfx950 transposing LDS read
// ds_read_b64_tr_b16 (inside each 16-lane group, lane i slot q receives element
// i % 4 of the 8 bytes that lane 4 q + i / 4 addressed); fp32 gathers.
template <class E>
__device__ __forceinline__ typename Tr<E>::frag tr_frag(const E *M, int ld, int row0, int colbase,
                                                        bool p32, int a, int li, int lg);
typedef short i16x4 __attribute__((ext_vector_type(4)));
template <>
__device__ __forceinline__ Tr<uint16_t>::frag tr_frag<uint16_t>(const uint16_t *M, int ld, int row0,
                                                                int colbase, bool p32, int a, int li,
                                                                int lg) {
    const int row = row0 + 8 * lg + (li >> 2);
    const int col = p32 ? colbase + 8 * (li & 3) + 4 * a : colbase + 4 * (li & 3);
    typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(M + row * ld + col));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4 *)(M + (row + 4) * ld + col));
    return Tr<uint16_t>::cat(__builtin_bit_cast(u32x2, lo), __builtin_bit_cast(u32x2, hi));
}
template <>
__device__ __forceinline__ Tr<float>::frag tr_frag<float>(const float *M, int ld, int row0, int colbase,
                                                          bool p32, int a, int li, int lg) {
    const int col = p32 ? colbase + p32_row(a, li) : colbase + li;
    Tr<float>::frag f;
#pragma unroll
    for (int q = 0; q < 8; ++q) f[q] = M[(row0 + 8 * lg + q) * ld + col];
    return f;
}

// Workgroup barrier that orders LDS only: outstanding global loads and stores
// stay in flight across it (a plain __syncthreads() also drains them).  Use it
// only where waves communicate through LDS.
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

template <int N> __device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N <= 63, "vmcnt range");
    asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Workgroup barrier for waves that communicate through LDS while asynchronous
// global->LDS copies are in flight: waits for this wave's LDS accesses only
// (a workgroup fence would also wait for the copies).
__device__ __forceinline__ void lds_only_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Single 16x16x4 fp32 MFMA step used by the fp32 triangular solve.
__device__ __forceinline__ f32x4 mma_f32_k4(float a, float b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

}  // namespace gdn
