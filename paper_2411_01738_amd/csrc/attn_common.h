// Device helpers shared by the bf16 attention kernels (attn_bf16.hip and
// attn_w64.hip): vector types, buffer resources, loads into LDS, wait
// counters, the launch arguments of one attention launch, and small lane
// exchanges.  Included inside namespace xdit::{anonymous} of each kernel
// source.
#pragma once

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef short s16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

constexpr uint32_t kOOB = 0x80000000u;  // offset past any buffer's range: reads 0, writes dropped
constexpr int kRsrcFlags = 0x00020000;  // raw buffer, 32-bit data format
constexpr float kRescaleLog2 = 8.0f;    // raise the reference max only beyond 2^8 growth
constexpr int kLdsBytes = 160 * 1024;   // LDS per CU on gfx950

struct Args {
    const uint16_t* q;
    const uint16_t* k;
    const uint16_t* v;
    const uint16_t* fk;
    const uint16_t* fv;
    uint16_t* wk;
    uint16_t* wv;
    uint16_t* out;
    float* lse;
    int B, H, Nq, Nk, q_tiles;
    int off0, len0, off1, len1;  // fresh ranges (fresh rows: range 0's, then range 1's)
    int sa0, sn0, sa1, sn1;      // tiles [sa, sa + sn) hold rows of fresh range 0 / 1
    float c2;  // softmax scale * log2(e)
    int accum;  // merge into the running (out, lse) instead of overwriting them
    // Work partition.  A pair is one query tile of one (batch, head), pair
    // index bh * q_tiles + qt; its sweep is T K/V tiles (T >= 1); the units
    // (pair, tile) are counted in pair-major order, pairs * T of them.  In a
    // partitioned launch the first G1 workgroups sweep pairs 0..G1-1 whole,
    // one each; the units of the other pairs, [G1 * T, units), are split
    // into G2 = gridDim.x - G1 contiguous ranges, one per further
    // workgroup.  A workgroup walks its range as segments, one per pair it
    // touches.  A segment over a whole sweep writes out (and lse); any other
    // writes its normalised partial O and its LSE to slot j (the range's
    // first segment) or G2 + j (its last) of `part`, j = the range index,
    // for the fix-up.
    int T;
    int64_t units;
    int G1;
    float* part;
};

typedef __amdgpu_buffer_rsrc_t Rsrc;

__device__ __forceinline__ Rsrc rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, kRsrcFlags);
}
__device__ __forceinline__ u32x4 bload(Rsrc r, uint32_t off) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0);
}
__device__ __forceinline__ void bstore(Rsrc r, uint32_t off, u32x4 x) {
    __builtin_amdgcn_raw_buffer_store_b128(x, r, off, 0, 0);
}
// 16 bytes per lane from global memory straight into LDS: lane l's bytes
// land at dst + 16*l (dst must be the same in every lane).
__device__ __forceinline__ void dma16(Rsrc r, void* dst, uint32_t off) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)dst, 16, off, 0, 0, 0);
}

// Wait until at most N vector-memory operations of this wave are in flight
// (LDS and export counters left unconstrained).
template <int N>
__device__ __forceinline__ void wait_vmem() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// f(integral_constant<int, I>) for I = B .. E-1, unrolled at compile time.
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    if constexpr (B < E) {
        f(std::integral_constant<int, B>{});
        static_for<B + 1, E>(f);
    }
}

// Transposing LDS read (ds_read_b64_tr_b16) at byte address a + OFF, issued
// without a wait: the caller waits with lds_wait_upto() before using the result.
// Written as inline assembly so that the compiler does not also drain the
// in-flight tile loads before it (it cannot tell that they target other LDS
// bytes).
template <int OFF>
__device__ __forceinline__ u32x2 tr_read(uint32_t a) {
    static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
    u32x2 r;
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(a), "i"(OFF));
    return r;
}
// An ordinary LDS load at byte address a: the compiler places its wait and
// folds a constant part of a into the instruction's offset.
template <typename T>
__device__ __forceinline__ T lds_ld(uint32_t a) {
    return *reinterpret_cast<const __attribute__((address_space(3))) T*>(a);
}
// A 16-byte LDS read at byte address a + OFF, issued without a wait (the
// caller waits for it by lgkmcnt).
template <int OFF>
__device__ __forceinline__ u32x4 lds_b128(uint32_t a) {
    static_assert(OFF >= 0 && OFF < 65536, "ds offset range");
    u32x4 r;
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(a), "i"(OFF));
    return r;
}
template <int N>
__device__ __forceinline__ void lgkm_wait_v4(u32x4& r) {
    static_assert(N >= 0 && N <= 15, "lgkmcnt range");
    asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N));
    asm volatile("" : "+v"(r));
}
// Wait until at most N LDS reads of this wave are in flight (they complete
// in issue order), then mark the registers of the reads that were covered.
__device__ __forceinline__ void lds_hold_one(u32x2& r) { asm volatile("" : "+v"(r)); }
template <int N, typename... R>
__device__ __forceinline__ void lds_wait_upto(R&... r) {
    static_assert(N >= 0, "lgkmcnt range");
    asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(N < 15 ? N : 15));
    (lds_hold_one(r), ...);
}
// Key of S^T row x (0..31) of a 32-key block: x = 16a + 8e + 4h + j is key
// 16a + 4j + 2e + h when PERM, key x otherwise.
template <bool PERM>
__device__ __forceinline__ int krow(int x) {
    if constexpr (PERM) return (x & 16) + 4 * (x & 3) + 2 * ((x >> 3) & 1) + ((x >> 2) & 1);
    else return x;
}

__device__ __forceinline__ int xcd_remap(int pid, int total) {
    const int per = total >> 3, rem = total & 7;
    const int xcd = pid & 7, loc = pid >> 3;
    return xcd * per + (xcd < rem ? xcd : rem) + loc;
}

// Two floats to a packed bf16 pair (round to nearest even): one v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
    typedef float f32x2_t __attribute__((ext_vector_type(2)));
    typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t));
}

// x combined with its value in the other 32-lane half (lane l <-> l ^ 32);
// the result is bit-identical in both lanes of a pair.
__device__ __forceinline__ float halves_max(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float halves_sum(float x) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

