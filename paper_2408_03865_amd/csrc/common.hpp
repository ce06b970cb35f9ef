// common.hpp -- device helpers shared by the gfx950 kernels: storage types,
// vector loads/stores with ragged tails, and DPP lane moves for wave64 rows.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace pm {

// ---------------------------------------------------------------------------
// storage types: float, or bf16 held as its 16-bit pattern
// ---------------------------------------------------------------------------
struct bf16_t {
    uint16_t bits;
};

typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// two floats -> two bf16 packed in one word, round to nearest even (v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
    f32x2 v = {a, b};
    bf16x2 r = __builtin_convertvector(v, bf16x2);
    return __builtin_bit_cast(uint32_t, r);
}

template <typename T> struct Storage;

template <> struct Storage<float> {
    static constexpr int kBytes = 4;
    static constexpr int kPerVec = 4;     // elements per 16-byte vector
    __device__ static float load1(const float* p) { return *p; }
    __device__ static void store1(float* p, float v) { *p = v; }
    __device__ static void unpack(const u32x4& w, float* v) {
        v[0] = __uint_as_float(w.x); v[1] = __uint_as_float(w.y);
        v[2] = __uint_as_float(w.z); v[3] = __uint_as_float(w.w);
    }
    __device__ static u32x4 pack(const float* v) {
        u32x4 w = {__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]),
                   __float_as_uint(v[3])};
        return w;
    }
};

template <> struct Storage<bf16_t> {
    static constexpr int kBytes = 2;
    static constexpr int kPerVec = 8;
    __device__ static float load1(const bf16_t* p) { return __uint_as_float((uint32_t)p->bits << 16); }
    __device__ static void store1(bf16_t* p, float v) {
        p->bits = (uint16_t)(pack_bf16x2(v, 0.0f) & 0xffffu);
    }
    __device__ static void unpack(const u32x4& w, float* v) {
        v[0] = bf16_lo(w.x); v[1] = bf16_hi(w.x); v[2] = bf16_lo(w.y); v[3] = bf16_hi(w.y);
        v[4] = bf16_lo(w.z); v[5] = bf16_hi(w.z); v[6] = bf16_lo(w.w); v[7] = bf16_hi(w.w);
    }
    __device__ static u32x4 pack(const float* v) {
        u32x4 w = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]), pack_bf16x2(v[4], v[5]),
                   pack_bf16x2(v[6], v[7])};
        return w;
    }
};

// Load K consecutive elements starting at row[l0] (K a multiple of the vector width),
// converting to float; elements at or beyond L read as `fill`.  `vec` says the row
// base is 16-byte aligned and L is a multiple of the vector width.
// With FULL the caller guarantees l0 + K <= L and vector alignment, so the loads are
// unconditional (no control flow: the compiler can batch them and defer the waits).
template <typename T, int K, bool FULL = false>
__device__ __forceinline__ void load_run(const T* __restrict__ row, int64_t l0, int64_t L, bool vec,
                                         float* v, float fill = 0.0f) {
    constexpr int PV = Storage<T>::kPerVec;
    static_assert(K % PV == 0, "K must be a multiple of the vector width");
    if (FULL || (vec && l0 + K <= L)) {
#pragma unroll
        for (int i = 0; i < K / PV; ++i) {
            const u32x4 w = *reinterpret_cast<const u32x4*>(row + l0 + i * PV);
            Storage<T>::unpack(w, v + i * PV);
        }
    } else {
#pragma unroll
        for (int i = 0; i < K; ++i) v[i] = (l0 + i < L) ? Storage<T>::load1(row + l0 + i) : fill;
    }
}

// K consecutive elements at row[l0] as raw 16-byte vectors (l0 + K <= L, vector
// aligned), converted later by unpack_run: the loads can be issued well before the
// values are needed, e.g. ahead of a barrier.
template <typename T, int K>
struct RawRun {
    u32x4 w[K / Storage<T>::kPerVec];
};
template <typename T, int K>
__device__ __forceinline__ RawRun<T, K> load_raw(const T* __restrict__ row, int64_t l0) {
    constexpr int PV = Storage<T>::kPerVec;
    RawRun<T, K> r;
#pragma unroll
    for (int i = 0; i < K / PV; ++i) r.w[i] = *reinterpret_cast<const u32x4*>(row + l0 + i * PV);
    return r;
}
// The same, non-temporal: for inputs read once, so that they do not take cache space
// from inputs that are read again.
template <typename T, int K>
__device__ __forceinline__ RawRun<T, K> load_raw_nt(const T* __restrict__ row, int64_t l0) {
    constexpr int PV = Storage<T>::kPerVec;
    RawRun<T, K> r;
#pragma unroll
    for (int i = 0; i < K / PV; ++i)
        r.w[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(row + l0 + i * PV));
    return r;
}
template <typename T, int K>
__device__ __forceinline__ void unpack_run(const RawRun<T, K>& r, float* v) {
    constexpr int PV = Storage<T>::kPerVec;
#pragma unroll
    for (int i = 0; i < K / PV; ++i) Storage<T>::unpack(r.w[i], v + i * PV);
}

// Store K consecutive elements (rounding to T) at row[l0]; elements beyond L are dropped.
// When a lane's K elements are one 16-byte vector, a wave's store covers 1 KB of
// consecutive bytes, and the store is non-temporal: every output here is streamed
// out once, and keeping it out of the caches leaves them to the inputs that are read
// again.  With more vectors per lane each store covers every other 16 bytes of its
// range; such partial lines are left to the caches to combine unless NT says
// otherwise (non-temporal, the fp32 conv backward's dx ran 40% slower, while the fp32
// scan backward's outputs gained 2%).
template <typename T, int K, bool FULL = false, bool NT = (K == Storage<T>::kPerVec)>
__device__ __forceinline__ void store_run(T* __restrict__ row, int64_t l0, int64_t L, bool vec,
                                          const float* v) {
    constexpr int PV = Storage<T>::kPerVec;
    if (FULL || (vec && l0 + K <= L)) {
#pragma unroll
        for (int i = 0; i < K / PV; ++i) {
            u32x4* dst = reinterpret_cast<u32x4*>(row + l0 + i * PV);
            if constexpr (NT) __builtin_nontemporal_store(Storage<T>::pack(v + i * PV), dst);
            else *dst = Storage<T>::pack(v + i * PV);
        }
    } else {
#pragma unroll
        for (int i = 0; i < K; ++i)
            if (l0 + i < L) Storage<T>::store1(row + l0 + i, v[i]);
    }
}

// ---------------------------------------------------------------------------
// DPP lane moves inside 16-lane rows (bound_ctrl off: a lane whose source is
// outside its row keeps `old`)
// ---------------------------------------------------------------------------
enum : int {
    kRowShl1 = 0x101,
    kRowShr1 = 0x111,
    kNewBcast0 = 0x150,
    kNewBcast15 = 0x15f,
};
__host__ __device__ constexpr int row_shl(int n) { return 0x100 + n; }
__host__ __device__ constexpr int row_shr(int n) { return 0x110 + n; }

template <int CTRL>
__device__ __forceinline__ float dpp(float old, float v) {
    return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, old),
                                                                  __builtin_bit_cast(int, v), CTRL,
                                                                  0xf, 0xf, false));
}

// Fused DPP arithmetic inside 16-lane rows.  The compiler does not fold a DPP
// move into a VOP2 consumer when the move's `old` operand is a constant, so these
// are written directly; a lane whose source is outside its row is disabled and
// keeps its value, which is the identity of each operation.  gfx9 needs two wait
// states between a VALU write of a VGPR and a DPP read of it: each op starts with
// `s_nop 1`, and each sequence below ends with one, so DPP reads issued by the
// surrounding compiler-generated code are covered too.
#define PM_DPP_OPS(NAME, CTRL)                                                              \
    __device__ __forceinline__ void mul_##NAME(float& x) { /* x = x[src] * x */            \
        asm("s_nop 1\n\tv_mul_f32_dpp %0, %0, %0 " CTRL                           \
                     " row_mask:0xf bank_mask:0xf"                                \
                     : "+v"(x));                                                            \
    }                                                                                       \
    __device__ __forceinline__ void fmac_##NAME(float& h, float p) { /* h = h[src] * p + h */ \
        asm("s_nop 1\n\tv_fmac_f32_dpp %0, %0, %1 " CTRL                          \
                     " row_mask:0xf bank_mask:0xf"                                \
                     : "+v"(h)                                                              \
                     : "v"(p));                                                             \
    }                                                                                       \
    __device__ __forceinline__ void add_##NAME(float& x) { /* x = x[src] + x */            \
        asm("s_nop 1\n\tv_add_f32_dpp %0, %0, %0 " CTRL                           \
                     " row_mask:0xf bank_mask:0xf"                                \
                     : "+v"(x));                                                            \
    }
PM_DPP_OPS(shr1, "row_shr:1")
PM_DPP_OPS(shr2, "row_shr:2")
PM_DPP_OPS(shr4, "row_shr:4")
PM_DPP_OPS(shr8, "row_shr:8")
PM_DPP_OPS(shl1, "row_shl:1")
PM_DPP_OPS(shl2, "row_shl:2")
PM_DPP_OPS(shl4, "row_shl:4")
PM_DPP_OPS(shl8, "row_shl:8")
#undef PM_DPP_OPS

// Inclusive scan, inside each 16-lane row, of the affine maps x -> P x + H.
// Forward (towards higher lanes): lane j ends with the composition of lanes 0..j
// (lane j's map applied last).  Reverse: lane j ends with the composition of
// lanes 15..j (lane j's map applied last).
__device__ __forceinline__ void dpp_tail_nop(float& x) { asm("s_nop 1" : "+v"(x)); }

__device__ __forceinline__ void row_scan_up(float& P, float& H) {
    fmac_shr1(H, P); mul_shr1(P);
    fmac_shr2(H, P); mul_shr2(P);
    fmac_shr4(H, P); mul_shr4(P);
    fmac_shr8(H, P); mul_shr8(P);
    dpp_tail_nop(P);
}
__device__ __forceinline__ void row_scan_down(float& P, float& H) {
    fmac_shl1(H, P); mul_shl1(P);
    fmac_shl2(H, P); mul_shl2(P);
    fmac_shl4(H, P); mul_shl4(P);
    fmac_shl8(H, P); mul_shl8(P);
    dpp_tail_nop(P);
}
// Both scans at once: the forward scan of (P, H) and the reverse scan of (Pr, Hr),
// interleaved so that every DPP read comes at least three instructions after the
// write of its source.  No wait states are needed inside, and each chain hides
// the other's DPP latency.
#define PM_UD_LEVEL(N)                                                        \
    "v_fmac_f32_dpp %1, %1, %0 row_shr:" #N " row_mask:0xf bank_mask:0xf\n\t" \
    "v_fmac_f32_dpp %3, %3, %2 row_shl:" #N " row_mask:0xf bank_mask:0xf\n\t" \
    "v_mul_f32_dpp %0, %0, %0 row_shr:" #N " row_mask:0xf bank_mask:0xf\n\t"  \
    "v_mul_f32_dpp %2, %2, %2 row_shl:" #N " row_mask:0xf bank_mask:0xf\n\t"
__device__ __forceinline__ void row_scan_up_down(float& P, float& H, float& Pr, float& Hr) {
    asm("s_nop 1\n\t" PM_UD_LEVEL(1) PM_UD_LEVEL(2) PM_UD_LEVEL(4) PM_UD_LEVEL(8) "s_nop 1"
        : "+v"(P), "+v"(H), "+v"(Pr), "+v"(Hr));
}
#undef PM_UD_LEVEL

// Sum over the 16 lanes of a row, delivered to lane 15.
__device__ __forceinline__ float row_sum_to_15(float x) {
    add_shr1(x); add_shr2(x); add_shr4(x); add_shr8(x);
    dpp_tail_nop(x);
    return x;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }
__device__ __forceinline__ float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// softplus(s) = ln(1 + e^s) = max(s, 0) + ln(1 + x), x = e^-|s| in (0, 1], without a
// branch.  With u = fl(1 + x), the rounding error e = x - (u - 1) is exact (u - 1 and
// x - (u - 1) are exact differences: Sterbenz's lemma), and ln(1 + x) = ln(u) + ln(1 + e/u).
// Replacing ln(1 + e/u) by e errs by at most |e| (1 - 1/u) <= 2^-24 x, while
// ln(1 + x) >= x ln 2: under 1e-7 relative for every s.  For s > 20 the result rounds to
// s itself, the usual threshold's value.
__device__ __forceinline__ float softplus_f(float s) {
    const float x = fast_exp2(-fabsf(s) * kLog2e);
    const float u = 1.0f + x;
    const float e = x - (u - 1.0f);
    return fmaxf(s, 0.0f) + fmaf(fast_log2(u), kLn2, e);
}
// d softplus(s)/ds = sigmoid(s) = e^(s - softplus(s)), from softplus(s) already at hand:
// one exp, and exactly 1 where softplus(s) rounded to s.
__device__ __forceinline__ float softplus_grad_f(float s, float sp) { return fast_exp2((s - sp) * kLog2e); }
__device__ __forceinline__ float sigmoid_f(float v) { return fast_rcp(1.0f + fast_exp2(-v * kLog2e)); }

// Flat wave lane id and the lane's position inside its 16-lane row.
__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }

}  // namespace pm
