// Device-side building blocks shared by the dmlnn kernels (gfx950 / CDNA4).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace dmlnn {

typedef double d4 __attribute__((ext_vector_type(4)));
typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kWave = 64;

// One 16x16x4 matrix-core step, D = A(16x4) * B(4x16) + C, per element type.
//
// Operand lanes (both types): lane l holds A[l % 16][l / 16] and B[l / 16][l % 16].
// Accumulator lanes differ between the two instructions on gfx950 (measured):
//   f64: item r of lane l is D[l / 16 + 4 r][l % 16]
//   f32: item r of lane l is D[4 (l / 16) + r][l % 16]
template <typename T>
struct Mfma;

template <>
struct Mfma<double> {
    typedef d4 acc_t;
    static __device__ __forceinline__ acc_t zero() { return acc_t{0.0, 0.0, 0.0, 0.0}; }
    static __device__ __forceinline__ acc_t mma(double a, double b, acc_t c)
    {
        return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ int row(int lane, int r) { return (lane >> 4) + 4 * r; }
};

template <>
struct Mfma<float> {
    typedef f4 acc_t;
    static __device__ __forceinline__ acc_t zero() { return acc_t{0.f, 0.f, 0.f, 0.f}; }
    static __device__ __forceinline__ acc_t mma(float a, float b, acc_t c)
    {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    static __device__ __forceinline__ int row(int lane, int r) { return 4 * (lane >> 4) + r; }
};

__device__ __forceinline__ int lane_id() { return threadIdx.x & (kWave - 1); }
// Wave index, made visibly wave-uniform so index math on it stays scalar.
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); }

// The value of x, hidden from the optimiser: index math derived from it inside
// a loop is recomputed per iteration instead of being hoisted into registers
// that stay live across the loop (which would spill next to the accumulators).
__device__ __forceinline__ int opaque(int x)
{
    asm volatile("" : "+v"(x));
    return x;
}

// floor(n / d) for 0 <= n < 2^16 and 1 <= d < 2^16, with magic = ceil(2^32 / d)
// computed on the host as a 64-bit value (2^32 itself for d = 1).  n * magic / 2^32
// exceeds n / d by less than n / 2^32, which is below 1/d when n * d < 2^32, so
// the floor is exact.
__device__ __forceinline__ int div_magic(int n, unsigned long long magic)
{
    return (int)(((unsigned long long)(unsigned)n * magic) >> 32);
}

// floor(n / d) for 0 <= n < 2^22 and 1 <= d < 2^22, with rcp = 1.0f / d.  The
// float product n * rcp is within a relative 2^-22 of n / d (rcp and the
// product each round once), i.e. within 1 of it, so its truncation is off by
// at most one either way and one correction step makes it exact.
__device__ __forceinline__ int div_small(int n, int d, float rcp)
{
    int q = (int)((float)n * rcp);
    const int r = n - q * d;
    q += (r >= d) - (r < 0);
    return q;
}

inline unsigned long long host_magic(int d)
{
    return (0x100000000ull + (unsigned long long)d - 1ull) / (unsigned long long)d;
}

// Wave-uniform "is every lane's value zero" test (wavefront ballot).
template <typename T>
__device__ __forceinline__ bool wave_all_zero(T v)
{
    return __builtin_amdgcn_ballot_w64(v != T(0)) == 0ull;
}

template <typename T>
__device__ __forceinline__ T relu_if(T v, int relu)
{
    return (relu && !(v > T(0))) ? T(0) : v;
}

// Gradient of a conv's output taken straight from the backward of a following
// relu -> max-pool (vertical fusion: the routed gradient is never stored).
// Windows PH x PW at stride PS >= PH, PW without padding do not overlap, so
// output cell (oy, ox) of filter f lies in at most one window (py, px); it
// receives that window's gradient when it is the window's argmax (the in-row
// index f*Q + oy*Wout + ox) and the pooled value is positive (the routed cell
// holds the pooled value, so that is its relu mask).
struct PoolSrc {
    const void *dpool;       // [N][F][Hp][Wp] gradient of the pooled output
    const int32_t *argmax;   // [N][F][Hp][Wp] in-row argmax of each window
    const void *pooled;      // [N][F][Hp][Wp] pooled values
    int PH, PW, PS, Hp, Wp;
    unsigned long long magic_ps;  // host_magic(PS); oy, ox < 2^16 (checked on the host)
};

// Branch-free, so the loads of several cells issue together (a load under a
// divergent branch is waited for where the branch ends): a cell no window
// covers reads its plane's first window and is dropped.  (n, f) must name a
// plane and (oy, ox) lie in [0, 2^16).
template <typename T>
__device__ __forceinline__ T pool_src_grad(const PoolSrc &p, int n, int F, int f, int Q, int Wout,
                                           int oy, int ox)
{
    const int py = div_magic(oy, p.magic_ps), px = div_magic(ox, p.magic_ps);
    const bool in = oy - py * p.PS < p.PH && ox - px * p.PS < p.PW && py < p.Hp && px < p.Wp;
    const size_t o = ((size_t)n * F + f) * p.Hp * p.Wp + (in ? (size_t)py * p.Wp + px : 0);
    const T d = reinterpret_cast<const T *>(p.dpool)[o];
    const int32_t am = p.argmax[o];
    const T pv = reinterpret_cast<const T *>(p.pooled)[o];
    return (in && am == f * Q + oy * Wout + ox && pv > T(0)) ? d : T(0);
}

// Blocks are dispatched round-robin over the 8 XCDs (block b runs on XCD b % 8).
// Renumber so that logically consecutive blocks share an XCD (and its L2): with
// m = floor(n / 8), block b < 8m gets logical id (b % 8) * m + b / 8; the last
// n % 8 blocks keep their own number.
__device__ __forceinline__ int xcd_logical_block(int b, int nblocks)
{
    const int m = nblocks >> 3;
    if (b >= 8 * m) return b;
    return (b & 7) * m + (b >> 3);
}

// ---- direct global -> LDS loads (LDS DMA) ----------------------------------
// A raw buffer resource: 64-bit base, byte range (loads at offsets >= range
// return 0 without touching memory), and the gfx9-family format word.
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;

extern "C" __device__ void llvm_amdgcn_raw_buffer_load_lds(i32x4 rsrc, lds_void *lds, int size,
                                                           int voffset, int soffset, int offset,
                                                           int aux)
    __asm("llvm.amdgcn.raw.buffer.load.lds");

__device__ __forceinline__ i32x4 buffer_rsrc(const void *base, unsigned range_bytes)
{
    const unsigned long long a = (unsigned long long)base;
    i32x4 r;
    r.x = __builtin_amdgcn_readfirstlane((int)(a & 0xffffffffu));
    r.y = __builtin_amdgcn_readfirstlane((int)(a >> 32));
    r.z = __builtin_amdgcn_readfirstlane((int)range_bytes);
    r.w = 0x00020000;
    return r;
}

// Out-of-range voffset: the load writes zeros to LDS.
constexpr int kDmaZero = (int)0x80000000u;

// One wave-wide DMA of 4 bytes per lane: lane i's dword from byte offset
// voffset + soffset of the buffer lands at lds_base + 4 i (lds_base wave-uniform).
__device__ __forceinline__ void dma_dword(i32x4 rsrc, void *lds_base, int voffset, int soffset)
{
    llvm_amdgcn_raw_buffer_load_lds(rsrc, (lds_void *)lds_base, 4, voffset, soffset, 0, 0);
}

// The same with 16 bytes per lane: lane i's four dwords land at lds_base + 16 i.
// The source needs only 4-byte alignment, and the range test is per dword (a
// lane straddling the end of the range loads its dwords below it, zeros above).
__device__ __forceinline__ void dma_x4(i32x4 rsrc, void *lds_base, int voffset, int soffset)
{
    llvm_amdgcn_raw_buffer_load_lds(rsrc, (lds_void *)lds_base, 16, voffset, soffset, 0, 0);
}

__device__ __forceinline__ void wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Kernels asking for more than 64 KiB of dynamic LDS must opt in (gfx950 has
// 160 KiB per CU).
template <typename Kernel>
inline hipError_t allow_dynamic_lds(Kernel kernel, size_t bytes)
{
    if (bytes <= 64 * 1024) return hipSuccess;
    // The attribute persists per device and kernel: set it once per (device,
    // kernel) for the largest size asked so far (a per-thread cache; the small
    // LeNet-sized launches otherwise pay the call every time).
    struct Entry {
        int dev;
        const void *k;
        size_t bytes;
    };
    thread_local Entry cache[32];
    thread_local int used = 0;
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return hipErrorInvalidDevice;
    const void *k = reinterpret_cast<const void *>(kernel);
    int slot = -1;
    for (int i = 0; i < used; ++i)
        if (cache[i].dev == dev && cache[i].k == k) {
            if (cache[i].bytes >= bytes) return hipSuccess;
            slot = i;
            break;
        }
    const hipError_t e =
        hipFuncSetAttribute(k, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e != hipSuccess) return e;
    if (slot < 0) {
        slot = used < 32 ? used++ : 0;
        cache[slot].dev = dev;
        cache[slot].k = k;
    }
    cache[slot].bytes = bytes;
    return hipSuccess;
}

// Resident blocks of `kernel` per CU for `lds` bytes of dynamic LDS, and the CU
// count of the current device (both cached per device and LDS size by callers).
template <typename Kernel>
inline int resident_slots(Kernel kernel, int threads, size_t lds)
{
    struct Entry {
        int dev, threads, slots;
        const void *k;
        size_t lds;
    };
    thread_local Entry cache[32];
    thread_local int used = 0, next = 0;
    int dev = 0, cus = 0, per_cu = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    const void *k = reinterpret_cast<const void *>(kernel);
    for (int i = 0; i < used; ++i)
        if (cache[i].dev == dev && cache[i].k == k && cache[i].threads == threads &&
            cache[i].lds == lds)
            return cache[i].slots;
    if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
        return 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, threads, lds) != hipSuccess)
        return 0;
    Entry &c = cache[used < 32 ? used++ : (next++ & 31)];
    c = Entry{dev, threads, cus * per_cu, k, lds};
    return c.slots;
}

}  // namespace dmlnn
