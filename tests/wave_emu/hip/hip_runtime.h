// Host emulation of the HIP device environment used by the int8 screening
// kernels and the cell assignment kernel (test infrastructure only; the
// library never runs on the host).
// One host thread per lane; wave-collective operations (__shfl_xor, __any,
// readfirstlane, the int8 MFMA) exchange values through a per-wave barrier,
// __syncthreads is a per-block barrier, and blocks of a grid run one after
// another. Buffer loads honour the resource's byte range like the hardware
// (zero past the end); every other access is a plain host access, so
// AddressSanitizer reports any that leaves its allocation. Buffer loads with
// an LDS destination are asynchronous like on the device: the destination is
// poisoned when the load is issued and receives its data only at the next
// __syncthreads, so a read of it before that barrier sees the poison.
#pragma once
#include <stdint.h>
#include <string.h>
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <algorithm>
#include <atomic>
#include <barrier>
#include <thread>
#include <vector>
#include <functional>
#include <climits>
#include <array>
#include <mutex>

struct dim3 {
    unsigned x = 1, y = 1, z = 1;
    dim3() {}
    dim3(unsigned a, unsigned b = 1, unsigned c = 1) : x(a), y(b), z(c) {}
};
struct uint2 {
    unsigned x, y;
};
struct float4 {
    float x, y, z, w;
};
inline uint2 make_uint2(unsigned x, unsigned y) { return uint2{x, y}; }
inline float4 make_float4(float x, float y, float z, float w) { return float4{x, y, z, w}; }
struct longlong2 {
    long long x, y;
};
struct double2 {
    double x, y;
};
typedef int hipError_t;
typedef void *hipStream_t;
enum { hipSuccess = 0, hipErrorInvalidValue = 1 };
inline hipError_t hipGetLastError() { return hipSuccess; }

namespace emu {
extern thread_local dim3 tid, bid;
extern dim3 bdim, gdim;
struct Wave {
    std::barrier<> *bar;
    unsigned char buf[64][128];
};
struct DmaFlush {
    void operator()() noexcept;
};
struct Block {
    std::barrier<DmaFlush> *bar;
    Wave waves[16];
    std::mutex mu;
    std::vector<std::pair<char *, std::array<char, 16>>> pending;  // LDS writes of in-flight loads
    std::atomic<int> or_acc{0};  // __syncthreads_or
};
extern Block *blk;
// dynamic LDS of the running block (the launch's shared-memory bytes)
extern unsigned char *dyn_lds;
inline void DmaFlush::operator()() noexcept
{
    for (auto &p : blk->pending) memcpy(p.first, p.second.data(), 16);
    blk->pending.clear();
}
inline Wave &wave() { return blk->waves[tid.x / 64]; }
inline int lane() { return tid.x % 64; }
}  // namespace emu

#define threadIdx (emu::tid)
#define blockIdx (emu::bid)
#define blockDim (emu::bdim)
#define gridDim (emu::gdim)
#define __global__
#define __device__
#define __host__
#define __forceinline__ inline
#define __launch_bounds__(...)
#define __shared__ static
#define HIP_SYMBOL(x) (x)

inline int max(int a, int b) { return a > b ? a : b; }
inline int min(int a, int b) { return a < b ? a : b; }
inline unsigned max(unsigned a, unsigned b) { return a > b ? a : b; }
inline unsigned min(unsigned a, unsigned b) { return a < b ? a : b; }
inline long long max(long long a, long long b) { return a > b ? a : b; }
inline long long min(long long a, long long b) { return a < b ? a : b; }
inline long max(long a, long b) { return a > b ? a : b; }
inline long min(long a, long b) { return a < b ? a : b; }

inline void __syncthreads() { emu::blk->bar->arrive_and_wait(); }

// block-wide OR of p, a barrier like __syncthreads
inline int __syncthreads_or(int p)
{
    if (p) emu::blk->or_acc.fetch_or(1);
    __syncthreads();
    const int r = emu::blk->or_acc.load();
    __syncthreads();
    if (emu::tid.x == 0) emu::blk->or_acc.store(0);
    __syncthreads();
    return r;
}

template <typename T>
inline T __shfl_xor(T v, int m)
{
    static_assert(sizeof(T) <= 128, "");
    emu::Wave &w = emu::wave();
    memcpy(w.buf[emu::lane()], &v, sizeof(T));
    w.bar->arrive_and_wait();
    T r;
    memcpy(&r, w.buf[emu::lane() ^ m], sizeof(T));
    w.bar->arrive_and_wait();
    return r;
}

// v_permlane32_swap_b32 (the two results of the builtin): the upper 32
// lanes of the first operand trade places with the lower 32 lanes of the
// second (lane layout checked on the device).
struct PermlanePair {
    uint32_t v[2];
    uint32_t operator[](int i) const { return v[i]; }
};
inline PermlanePair __builtin_amdgcn_permlane32_swap(uint32_t old, uint32_t src, bool, bool)
{
    emu::Wave &w = emu::wave();
    const int l = emu::lane();
    const uint32_t in[2] = {old, src};
    memcpy(w.buf[l], in, sizeof in);
    w.bar->arrive_and_wait();
    PermlanePair r;
    memcpy(&r.v[0], w.buf[l < 32 ? l : l - 32] + (l < 32 ? 0 : 4), 4);
    memcpy(&r.v[1], w.buf[l < 32 ? l + 32 : l] + (l < 32 ? 0 : 4), 4);
    w.bar->arrive_and_wait();
    return r;
}

inline int __any(int p)
{
    emu::Wave &w = emu::wave();
    w.buf[emu::lane()][0] = p ? 1 : 0;
    w.bar->arrive_and_wait();
    int r = 0;
    for (int i = 0; i < 64; ++i) r |= w.buf[i][0];
    w.bar->arrive_and_wait();
    return r;
}

inline unsigned long long __ballot(int p)
{
    emu::Wave &w = emu::wave();
    w.buf[emu::lane()][0] = p ? 1 : 0;
    w.bar->arrive_and_wait();
    unsigned long long r = 0;
    for (int i = 0; i < 64; ++i) r |= (unsigned long long)w.buf[i][0] << i;
    w.bar->arrive_and_wait();
    return r;
}

template <typename T>
inline T __shfl(T v, int src)
{
    static_assert(sizeof(T) <= 128, "");
    emu::Wave &w = emu::wave();
    memcpy(w.buf[emu::lane()], &v, sizeof(T));
    w.bar->arrive_and_wait();
    T r;
    memcpy(&r, w.buf[src & 63], sizeof(T));
    w.bar->arrive_and_wait();
    return r;
}

inline int __ffsll(unsigned long long m) { return __builtin_ffsll((long long)m); }
inline int __popcll(unsigned long long m) { return __builtin_popcountll(m); }

// lanes below this one among the mask's low (lanes 0-31) and high (32-63) halves
inline unsigned __builtin_amdgcn_mbcnt_lo(unsigned m, unsigned acc)
{
    const int l = emu::lane();
    const unsigned below = l >= 32 ? 0xFFFFFFFFu : ((1u << l) - 1u);
    return acc + (unsigned)__builtin_popcount(m & below);
}
inline unsigned __builtin_amdgcn_mbcnt_hi(unsigned m, unsigned acc)
{
    const int l = emu::lane();
    const unsigned below = l < 32 ? 0u : ((1u << (l - 32)) - 1u);
    return acc + (unsigned)__builtin_popcount(m & below);
}

typedef int emu_i32x4 __attribute__((ext_vector_type(4)));
typedef int emu_i32x16 __attribute__((ext_vector_type(16)));

// v_mfma_i32_32x32x32_i8: lane l supplies A[l % 32][16 (l / 32) + 0..15] and
// B[k][l % 32] for k = 16 (l / 32) + 0..15; output register r of lane l is
// D[8 (r / 4) + 4 (l / 32) + r % 4][l % 32].
inline emu_i32x16 __builtin_amdgcn_mfma_i32_32x32x32_i8(emu_i32x4 a, emu_i32x4 b, emu_i32x16 c, int, int, int)
{
    emu::Wave &w = emu::wave();
    const int l = emu::lane();
    memcpy(w.buf[l], &a, 16);
    memcpy(w.buf[l] + 16, &b, 16);
    w.bar->arrive_and_wait();
    emu_i32x16 d;
    for (int r = 0; r < 16; ++r) {
        const int i = 8 * (r / 4) + 4 * (l / 32) + r % 4, j = l % 32;
        int s = 0;
        for (int k = 0; k < 32; ++k) {
            const int8_t av = (int8_t)w.buf[i + 32 * (k / 16)][k % 16];
            const int8_t bv = (int8_t)w.buf[j + 32 * (k / 16)][16 + k % 16];
            s += (int)av * (int)bv;
        }
        d[r] = (int)((uint32_t)s + (uint32_t)c[r]);
    }
    w.bar->arrive_and_wait();
    return d;
}

// v_dot4_i32_i8 without clamping: c + the dot of the four signed bytes
inline int __builtin_amdgcn_sdot4(int a, int b, int c, bool)
{
    for (int i = 0; i < 4; ++i) c += (int)(int8_t)(a >> (8 * i)) * (int)(int8_t)(b >> (8 * i));
    return c;
}

inline uint32_t __builtin_amdgcn_sad_u8(uint32_t a, uint32_t b, uint32_t c)
{
    for (int i = 0; i < 4; ++i) {
        const int x = (a >> (8 * i)) & 255, y = (b >> (8 * i)) & 255;
        c += x > y ? x - y : y - x;
    }
    return c;
}

struct __amdgpu_buffer_rsrc_t {
    const char *base;
    int64_t num;
};
inline __amdgpu_buffer_rsrc_t __builtin_amdgcn_make_buffer_rsrc(void *p, short, int num, int)
{
    return {(const char *)p, (int64_t)(unsigned)num};
}
// raw buffer loads: each dword past num_records reads zero (and is never touched)
inline emu_i32x4 __builtin_amdgcn_raw_buffer_load_b128(__amdgpu_buffer_rsrc_t r, int off, int soff, int)
{
    emu_i32x4 v = {0, 0, 0, 0};
    for (int i = 0; i < 4; ++i) {
        const int64_t o = (int64_t)(unsigned)off + soff + 4 * i;
        int t = 0;
        if (o + 4 <= r.num) memcpy(&t, r.base + o, 4);
        v[i] = t;
    }
    return v;
}
inline uint32_t __builtin_amdgcn_raw_buffer_load_b32(__amdgpu_buffer_rsrc_t r, int off, int soff, int)
{
    uint32_t v = 0;
    const int64_t o = (int64_t)(unsigned)off + soff;
    if (o + 4 <= r.num) memcpy(&v, r.base + o, 4);
    return v;
}
// 16-byte buffer load into LDS: lane l writes lds + 16 l; the data lands at
// the next __syncthreads, the destination holds a poison pattern until then
template <typename P>
inline void __builtin_amdgcn_raw_ptr_buffer_load_lds(__amdgpu_buffer_rsrc_t r, P lds, unsigned size, int off,
                                                     int soff, int ioff, int)
{
    if (size != 16) abort();
    const emu_i32x4 v = __builtin_amdgcn_raw_buffer_load_b128(r, off, soff, 0);
    char *dst = (char *)(uintptr_t)lds + ioff + 16 * emu::lane();
    std::array<char, 16> d;
    memcpy(d.data(), &v, 16);
    memset(dst, 0x5A, 16);
    std::lock_guard<std::mutex> g(emu::blk->mu);
    emu::blk->pending.push_back({dst, d});
}

inline int __builtin_amdgcn_readfirstlane(int v)
{
    emu::Wave &w = emu::wave();
    memcpy(w.buf[emu::lane()], &v, sizeof(int));
    w.bar->arrive_and_wait();
    int r;
    memcpy(&r, w.buf[0], sizeof(int));
    w.bar->arrive_and_wait();
    return r;
}

inline void __builtin_amdgcn_sched_barrier(int) {}
// the wave's lanes meet (every lane of the wave must come)
inline void __builtin_amdgcn_wave_barrier() { emu::wave().bar->arrive_and_wait(); }
// a compiler fence; the host's barriers already order the lanes' accesses
inline void __builtin_amdgcn_fence(int, const char *) {}

inline uint32_t __float_as_uint(float f)
{
    uint32_t u;
    memcpy(&u, &f, 4);
    return u;
}
inline float __uint_as_float(uint32_t u)
{
    float f;
    memcpy(&f, &u, 4);
    return f;
}
// double to float, rounded toward +infinity
inline float __double2float_ru(double x)
{
    float f = (float)x;
    if ((double)f < x) f = nextafterf(f, INFINITY);
    return f;
}

template <typename T>
inline T atomicAdd(T *p, T v) { return __atomic_fetch_add(p, v, __ATOMIC_SEQ_CST); }
inline unsigned long long atomicAdd(unsigned long long *p, unsigned long long v)
{
    return __atomic_fetch_add(p, v, __ATOMIC_SEQ_CST);
}
inline uint32_t atomicOr(uint32_t *p, uint32_t v) { return __atomic_fetch_or(p, v, __ATOMIC_SEQ_CST); }
inline uint32_t atomicMax(uint32_t *p, uint32_t v)
{
    uint32_t o = __atomic_load_n(p, __ATOMIC_SEQ_CST);
    while (o < v && !__atomic_compare_exchange_n(p, &o, v, false, __ATOMIC_SEQ_CST, __ATOMIC_SEQ_CST)) {}
    return o;
}

namespace emu {
// runs every block of the grid, one after another, with one host thread per
// lane; the lane threads are created once per launch and run every block
// (between blocks they wait at a launch barrier while the next block's LDS,
// barriers and state are set up afresh)
template <typename K, typename... A>
void launch(K kernel, dim3 grid, dim3 block, size_t shared_bytes, A... args)
{
    gdim = grid;
    bdim = block;
    const int nt = block.x;
    std::barrier<> start(nt + 1), done(nt + 1);
    bool quit = false;
    unsigned cur = 0;
    std::vector<std::thread> th;
    for (int t = 0; t < nt; ++t)
        th.emplace_back([&, t]() {
            tid = dim3(t);
            for (;;) {
                start.arrive_and_wait();
                if (quit) return;
                bid = dim3(cur);
                kernel(args...);
                done.arrive_and_wait();
            }
        });
    for (unsigned b = 0; b < grid.x; ++b) {
        // a fresh allocation per block, filled with a pattern, so that reads
        // of LDS the block did not write are seen and overruns are reported
        std::vector<unsigned char> lds(std::max<size_t>(shared_bytes, 1), 0xA5);
        dyn_lds = shared_bytes ? lds.data() : nullptr;
        Block B;
        std::barrier<DmaFlush> bb(nt);
        B.bar = &bb;
        std::vector<std::barrier<> *> wb;
        for (int w = 0; w < (nt + 63) / 64; ++w) {
            wb.push_back(new std::barrier<>(std::min(64, nt - 64 * w)));
            B.waves[w].bar = wb.back();
        }
        blk = &B;
        cur = b;
        start.arrive_and_wait();  // the block runs
        done.arrive_and_wait();   // every lane has finished it
        for (auto *p : wb) delete p;
    }
    quit = true;
    start.arrive_and_wait();
    for (auto &t : th) t.join();
}
}  // namespace emu
#define hipLaunchKernelGGL(k, g, b, sh, s, ...) emu::launch(k, g, b, (size_t)(sh), __VA_ARGS__)
