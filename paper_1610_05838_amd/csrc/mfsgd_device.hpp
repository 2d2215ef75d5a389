// mfsgd_device.hpp -- device building blocks of the gfx950 SGD-MF kernels.
//
// One SGD worker is one 64-lane wavefront.  A sample's feature rows (k values
// each) are spread over the lanes, E = KP/64 consecutive values per lane (at
// KP = 32 one value on each of the first 32 lanes), so every row is read and
// written with one coalesced vector access per lane.  The dot product is
// reduced across the wavefront with DPP row operations and the gfx950
// permlane swaps (no LDS, no barrier), which leaves the same sum in every
// lane.  Sample records are read 64 at a time (one per lane, streamed with
// non-temporal loads) and broadcast with v_readlane, so the row addresses are
// wave-uniform scalars.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mfsgd {

struct Sample {
    int32_t u;
    int32_t v;
    float r;
};
static_assert(sizeof(Sample) == 12, "a rating sample is two int32 and one float");

typedef _Float16 half_t;

template <typename T, int E>
struct VecT;
template <>
struct VecT<float, 1> { typedef float type; };
template <>
struct VecT<float, 2> { typedef float type __attribute__((ext_vector_type(2))); };
template <>
struct VecT<float, 4> { typedef float type __attribute__((ext_vector_type(4))); };
template <>
struct VecT<float, 8> { typedef float type __attribute__((ext_vector_type(8))); };
template <>
struct VecT<half_t, 1> { typedef half_t type; };
template <>
struct VecT<half_t, 2> { typedef half_t type __attribute__((ext_vector_type(2))); };
template <>
struct VecT<half_t, 4> { typedef half_t type __attribute__((ext_vector_type(4))); };
template <>
struct VecT<half_t, 8> { typedef half_t type __attribute__((ext_vector_type(8))); };

// Row geometry for a padded width KP.
template <int KP>
struct Geo {
    static constexpr int E = KP >= 64 ? KP / 64 : 1; // values per lane
    static constexpr int A = KP / E;                 // lanes that hold values (32 or 64)
};

// Loads and stores of one lane's E values of a feature row.
template <typename T, int E>
struct Row {
    typedef typename VecT<T, E>::type V;
    __device__ __forceinline__ static V ld(const T* p) { return *reinterpret_cast<const V*>(p); }
    __device__ __forceinline__ static void st(T* p, V v) { *reinterpret_cast<V*>(p) = v; }
    __device__ __forceinline__ static void widen(V v, float (&x)[E])
    {
        if constexpr (E == 1) {
            x[0] = (float)v;
        } else {
#pragma unroll
            for (int e = 0; e < E; ++e)
                x[e] = (float)v[e];
        }
    }
    // Binary16: every value is first a binary32 result in a register (the
    // empty asm keeps the compiler from fusing the conversion into the fma
    // that produced it, which would round once from the exact value instead),
    // then converted with round to nearest even; every kernel stores the same
    // bits for the same update.
    __device__ __forceinline__ static V narrow(const float (&x)[E])
    {
        V v;
        float y[E];
#pragma unroll
        for (int e = 0; e < E; ++e) {
            y[e] = x[e];
            if constexpr (sizeof(T) == 2)
                asm volatile("" : "+v"(y[e]));
        }
        if constexpr (E == 1) {
            v = (T)y[0];
        } else {
#pragma unroll
            for (int e = 0; e < E; ++e)
                v[e] = (T)y[e];
        }
        return v;
    }
    __device__ __forceinline__ static void load(const T* p, float (&x)[E]) { widen(ld(p), x); }
    __device__ __forceinline__ static void store(T* p, const float (&x)[E]) { st(p, narrow(x)); }
};

// Buffer addressing for rows whose per-lane part is one dword (binary16 at
// KP = 128, binary32 at KP <= 64): a descriptor for the whole matrix, the
// lane's byte offset in a VGPR (loop-invariant) and the row's byte offset in
// an SGPR, so a row access needs no vector address arithmetic.  Used only
// when every row offset fits 31 bits.  (The descriptor's fourth word selects
// 32-bit data, which raw loads and stores require; the record count is the
// largest, so the hardware range check never clips.)
struct Buf {
    __amdgpu_buffer_rsrc_t r;
    __device__ __forceinline__ explicit Buf(const void* base)
        : r(__builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, 0x7FFFFFFF, 0x00020000))
    {
    }
    template <typename V>
    __device__ __forceinline__ V ld(uint32_t voff, uint32_t soff) const
    {
        static_assert(sizeof(V) == 4, "one dword per lane");
        return __builtin_bit_cast(V, __builtin_amdgcn_raw_buffer_load_b32(r, (int)voff, (int)soff, 0));
    }
    template <typename V>
    __device__ __forceinline__ void st(V v, uint32_t voff, uint32_t soff) const
    {
        static_assert(sizeof(V) == 4, "one dword per lane");
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, (int)voff, (int)soff, 0);
    }
};

// ---------------------------------------------------------------------------
// Cross-lane sum over the 64 lanes; every lane receives the same value (each
// step adds a pair of lanes in both orders, and IEEE addition commutes).
// ---------------------------------------------------------------------------
// (bound_ctrl set: the patterns below read only valid lanes, and it lets the
// move fold into the add as one v_add_f32_dpp)
template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x)
{
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, true));
}

// Sum over each half of the wavefront on its own: lanes 0-31 receive the sum
// of lanes 0-31, lanes 32-63 that of lanes 32-63 (the first steps of
// wave_sum, which therefore adds the same terms in the same order).
__device__ __forceinline__ float half_sum(float x)
{
    x += dpp_mov<0xB1>(x);  // quad_perm [1,0,3,2]: pairs
    x += dpp_mov<0x4E>(x);  // quad_perm [2,3,0,1]: quads
    x += dpp_mov<0x141>(x); // row_half_mirror: 8 lanes
    x += dpp_mov<0x140>(x); // row_mirror: 16 lanes
    {
        // v_permlane16_swap: odd rows of the first operand trade places with
        // even rows of the second; with both operands x the two results hold,
        // lane for lane, the sums of rows {0,1} and {2,3} split over both.
        auto s = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
        x = __uint_as_float(s[0]) + __uint_as_float(s[1]);
    }
    return x;
}

__device__ __forceinline__ float wave_sum(float x)
{
    x = half_sum(x);
    {
        auto s = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
        x = __uint_as_float(s[0]) + __uint_as_float(s[1]);
    }
    return x;
}

__device__ __forceinline__ int lane_id() { return __builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)); }

// Agent-scope release that has finished before the next store issues: the
// fence writes this XCD's L2 back (buffer_wbl2), and the write-back counts on
// the vector memory counter like a store.  The fence's own wait for it is
// left out by this compiler's wait-count pass whenever no other memory
// operation is outstanding (it does not count the write-back), so a flag
// stored next could reach another XCD before the rows it publishes; the
// explicit wait keeps the order.
__device__ __forceinline__ void release_agent()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
    __builtin_amdgcn_s_waitcnt(0);
}

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ int64_t uniform64(int64_t x)
{
    uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
    uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// ---------------------------------------------------------------------------
// SplitMix64 (Steele, Lea, Flood 2014) in counter form: output number i of a
// generator whose state starts at s0 is the finaliser applied to
// s0 + (i+1) * golden-gamma.
// ---------------------------------------------------------------------------
__host__ __device__ __forceinline__ uint64_t sm64_at(uint64_t s0, uint64_t i)
{
    const uint64_t kGamma = 0x9E3779B97F4A7C15ull;
    uint64_t z = s0 + (i + 1ull) * kGamma;
    z ^= z >> 30;
    z *= 0xBF58476D1CE4E5B9ull;
    z ^= z >> 27;
    z *= 0x94D049BB133111EBull;
    z ^= z >> 31;
    return z;
}

// Stream keys used by the library: stream `tag` is output `tag` of the
// generator seeded with the user seed.
enum : uint64_t { kTagP = 1, kTagQ = 2, kTagColPerm = 16, kTagWaveOffset = 17 };
// global scheduling table: the draws of epoch t come from stream kTagTable + t
constexpr uint64_t kTagTable = uint64_t(1) << 40;

// Durstenfeld shuffle of 0..s-1: step i (from s-1 down to 1) swaps a[i]
// with a[j], j = high 32 bits of draw (s-1-i) times (i+1), shifted down 32.
__device__ __forceinline__ void shuffle_perm(uint64_t s0, int s, int* a)
{
    for (int i = 0; i < s; ++i)
        a[i] = i;
    for (int i = s - 1; i >= 1; --i) {
        uint64_t x = sm64_at(s0, (uint64_t)(s - 1 - i));
        int j = (int)(((x >> 32) * (uint64_t)(i + 1)) >> 32);
        int t = a[i];
        a[i] = a[j];
        a[j] = t;
    }
}

// Binary64 -> binary16 bits, round to nearest, ties to even, from the bit
// patterns: keep the 11 significant bits that binary16 has at this exponent
// (fewer below 2^-14) and round on the discarded remainder.
__device__ __forceinline__ uint16_t f64_to_f16_bits(double x)
{
    uint64_t b = (uint64_t)__double_as_longlong(x);
    uint16_t sgn = (uint16_t)((b >> 48) & 0x8000u);
    int ef = (int)((b >> 52) & 0x7ff);
    uint64_t frac = b & 0xFFFFFFFFFFFFFull;
    if (ef == 0x7ff)
        return (uint16_t)(sgn | (frac ? 0x7e00u : 0x7c00u));
    if (ef == 0)
        return sgn; // |x| < 2^-1022: far below the smallest binary16 subnormal
    int e = ef - 1023;
    if (e >= 16)
        return (uint16_t)(sgn | 0x7c00u);
    uint64_t sig = frac | (1ull << 52); // value = sig * 2^(e-52)
    int qexp = (e < -14 ? -14 : e) - 10; // exponent of one binary16 unit here
    int shift = qexp - (e - 52);         // >= 42
    if (shift >= 54)
        return sgn; // below half of the smallest subnormal
    uint64_t n = sig >> shift;
    uint64_t rem = sig & ((1ull << shift) - 1ull);
    uint64_t halfway = 1ull << (shift - 1);
    if (rem > halfway || (rem == halfway && (n & 1ull)))
        ++n;
    if (e < -14)
        return (uint16_t)(sgn | (uint16_t)n); // n == 1024 is the smallest normal
    if (n == 2048) {
        n = 1024;
        ++e;
    }
    if (e > 15)
        return (uint16_t)(sgn | 0x7c00u);
    return (uint16_t)(sgn | (uint16_t)((e + 15) << 10) | (uint16_t)(n - 1024));
}

template <typename T>
__device__ __forceinline__ T from_f64(double x);
template <>
__device__ __forceinline__ float from_f64<float>(double x)
{
    return (float)x; // v_cvt_f32_f64: round to nearest even
}
template <>
__device__ __forceinline__ half_t from_f64<half_t>(double x)
{
    uint16_t h = f64_to_f16_bits(x);
    return __builtin_bit_cast(half_t, h);
}

// Cross-XCD coherence of the one-address-space batch-Hogwild!: every `every`
// batches the XCD's leader wavefront writes its L2 back and invalidates it
// (an agent-scope release + acquire), which bounds how long an update made on
// one XCD stays invisible to the others; with `l1` the other wavefronts drop
// their CU's L1 at the same points.
struct CacheSync {
    int every;   // batches between flushes, 0 = never
    bool leader; // this wavefront flushes its XCD's L2
    bool l1;     // this wavefront invalidates its CU's L1
};

// Cross-XCD coherence of row updates in the one-address-space batch-Hogwild!.
// Each XCD's L2 is a write-back cache that the other XCDs do not see, so a
// row updated on one XCD and read on another while the line is still dirty
// in the first L2 is read stale, and whichever L2 writes the line back last
// discards the other's updates.  Rows stored with an agent-scope store
// (sc1) are written through to memory, where every XCD's next miss finds
// them.  Rows that hold a large share of the samples ("hot", one bit per row)
// keep write-back stores: their update rate would otherwise serialise on the
// one memory channel that holds them, and a row updated that often is
// over-determined, so losing part of its updates changes nothing measurable.
enum : int {
    kCohOff = 0,    // every store write-back (plain)
    kCohStore = 1,  // agent-scope stores for rows that are not hot
    kCohBoth = 2,   // ... and agent-scope loads for them
    kCohNT = 3,     // non-temporal stores for rows that are not hot
    kCohSys = 4,    // system-scope stores for rows that are not hot
};
struct Coherence {
    const uint32_t* hot_p; // bit u: row u of P is hot (nullptr: no row is)
    const uint32_t* hot_q; // bit v: row v of Q is hot
    bool p, q;             // apply the coherent policy to P's / Q's rows
};

__device__ __forceinline__ bool hot_bit(const uint32_t* __restrict__ bits, int i)
{
    return bits != nullptr && ((bits[(uint32_t)i >> 5] >> (i & 31)) & 1u) != 0;
}

template <int N>
struct UIntOf;
template <>
struct UIntOf<2> { typedef uint16_t type; };
template <>
struct UIntOf<4> { typedef uint32_t type; };
template <>
struct UIntOf<8> { typedef uint64_t type; };

// One lane's part of a row stored / loaded with the coherent policy COH.
template <int COH, typename V>
__device__ __forceinline__ void st_coh(V* p, V v)
{
    if constexpr (COH == kCohNT) {
        __builtin_nontemporal_store(v, p);
    } else {
        constexpr int scope = COH == kCohSys ? __HIP_MEMORY_SCOPE_SYSTEM : __HIP_MEMORY_SCOPE_AGENT;
        if constexpr (sizeof(V) <= 8) {
            typedef typename UIntOf<sizeof(V)>::type U;
            __hip_atomic_store(reinterpret_cast<U*>(p), __builtin_bit_cast(U, v), __ATOMIC_RELAXED, scope);
        } else {
            static_assert(sizeof(V) % 8 == 0, "rows are stored in 8-byte parts");
            uint64_t w[sizeof(V) / 8];
            __builtin_memcpy(w, &v, sizeof(V));
#pragma unroll
            for (int i = 0; i < (int)(sizeof(V) / 8); ++i)
                __hip_atomic_store(reinterpret_cast<uint64_t*>(p) + i, w[i], __ATOMIC_RELAXED, scope);
        }
    }
}

template <typename V>
__device__ __forceinline__ V ld_coh(const V* p)
{
    if constexpr (sizeof(V) <= 8) {
        typedef typename UIntOf<sizeof(V)>::type U;
        return __builtin_bit_cast(
            V, __hip_atomic_load(reinterpret_cast<const U*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    } else {
        uint64_t w[sizeof(V) / 8];
#pragma unroll
        for (int i = 0; i < (int)(sizeof(V) / 8); ++i)
            w[i] = __hip_atomic_load(reinterpret_cast<const uint64_t*>(p) + i, __ATOMIC_RELAXED,
                                     __HIP_MEMORY_SCOPE_AGENT);
        V v;
        __builtin_memcpy(&v, w, sizeof(V));
        return v;
    }
}

// Debug hooks of one epoch.
struct DebugSink {
    uint32_t* visits;     // per caller-array sample, or nullptr
    const int64_t* orig;  // planned position -> caller position, or nullptr
    int32_t* trace;       // batch -> worker, or nullptr
};

// ---------------------------------------------------------------------------
// One batch-Hogwild! worker (one wavefront).
//
// The worker's samples are the batches b = worker, worker+W, ... of f
// consecutive samples of S[0..nnz), in increasing b, each in array order;
// position q of this sequence is sample (worker + (q/f)*W)*f + q%f.  Rows of
// the next D-1 samples are requested before the current sample is written
// back; a requested row that an earlier, still-unwritten sample of this same
// worker updates is replaced by that sample's new value (nearest wins), so
// the worker's result is exactly the serial update of its sequence.
// Updates of other workers race (Hogwild!).
//
// The loop body has no branch around a memory instruction (a look-ahead past
// the end loads row 0 and is never used), so the compiler can keep all D
// samples' loads in flight with counted waits.
// ---------------------------------------------------------------------------
// by-value select (keeps the operands in registers)
template <typename V>
__device__ __forceinline__ V pick(bool c, V a, V b)
{
    return c ? a : b;
}

template <int KP, typename T, int D>
struct WorkerState {
    static constexpr int E = Geo<KP>::E;
    typedef typename VecT<T, E>::type V;
    V sp[D], sq[D]; // rows in flight, as loaded
    int su[D], sv[D];
    float sr[D];
    V hp[D], hq[D]; // rows of the last D samples, as stored
    int hu[D], hv[D];
    bool cp[D], cq[D]; // coherent policy for the rows in flight
};

// Atomic row updates: the change of every value is added with an L2 atomic
// (binary32 add, or packed binary16 add) instead of storing the new row, so
// concurrent updates of one row all take effect (Hogwild!'s model of
// component-wise atomic updates) rather than the last store winning.
//
// Binary32 rows of 2 or 4 values per lane are first transposed across the
// wavefront (ds_bpermute, no LDS storage) so that atomic instruction e adds
// values 64 e .. 64 e + 63 of the row, one per lane: each instruction then
// covers 256 contiguous bytes instead of the whole row with gaps.
// `row` points at value 0 of the row, `lane` is the lane index.
template <typename T, int E>
__device__ __forceinline__ void add_row_t(T* row, int lane, const float (&d)[E])
{
    static_assert(sizeof(T) == 4 && (E == 2 || E == 4), "transposed adds: binary32, 2 or 4 values per lane");
#pragma unroll
    for (int e = 0; e < E; ++e) {
        const int x = 64 * e + lane;         // value this lane adds in instruction e
        const int src = x / E, comp = x % E; // the lane that holds it, and where
        float v = 0.f;
#pragma unroll
        for (int c = 0; c < E; ++c) {
            const float y = __int_as_float(__builtin_amdgcn_ds_bpermute(src << 2, __float_as_int(d[c])));
            v = comp == c ? y : v;
        }
        __hip_atomic_fetch_add(reinterpret_cast<float*>(row) + x, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
}

template <typename T, int E>
__device__ __forceinline__ void add_row(T* p, const float (&d)[E])
{
    if constexpr (sizeof(T) == 4) {
#pragma unroll
        for (int e = 0; e < E; ++e)
            __hip_atomic_fetch_add(reinterpret_cast<float*>(p) + e, d[e], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    } else {
        static_assert(E % 2 == 0, "binary16 rows are added in pairs");
        typedef _Float16 h2 __attribute__((ext_vector_type(2)));
#pragma unroll
        for (int e = 0; e < E; e += 2) {
            h2 v = {(_Float16)d[e], (_Float16)d[e + 1]};
            __builtin_amdgcn_global_atomic_fadd_v2f16(reinterpret_cast<h2*>(p + e), v);
        }
    }
}

template <int KP, typename T, int D, bool DBG, bool SKIP = false, bool BUF = false, int COH = kCohOff,
          bool ATOM = false>
__device__ __forceinline__ void run_worker(const Sample* __restrict__ S, int64_t nnz, int64_t W, int64_t worker,
                                           int f, T* __restrict__ P, T* __restrict__ Q, float lr, float lp,
                                           float lq, const DebugSink dbg, const CacheSync sync = CacheSync{0, false, false},
                                           T* sink = nullptr, const Coherence coh = Coherence{nullptr, nullptr, false, false})
{
    constexpr int E = Geo<KP>::E;
    static_assert(!BUF || (!SKIP && sizeof(T) * E == 4), "buffer rows: one dword per lane, no store redirection");
    static_assert(COH == kCohOff || (!BUF && !SKIP), "coherent rows use global addressing");
    static_assert(!ATOM || (D == 1 && !BUF && !SKIP && COH != kCohStore && COH != kCohNT && COH != kCohSys),
                  "atomic updates: one sample in flight, global addressing");
    constexpr int A = Geo<KP>::A;
    typedef Row<T, E> R;
    static_assert(64 % D == 0 && D <= 32, "depth must divide 64");

    const int lane = lane_id();
    // lanes past the row width (KP = 32) mirror lane 0's address and never store
    const int col = (A == 64 || lane < A) ? lane * E : 0;
    const Buf bp(P), bq(Q);
    const uint32_t cb = (uint32_t)(col * sizeof(T));        // lane's byte offset in a row
    constexpr uint32_t kRowBytes = (uint32_t)(KP * sizeof(T));
    const bool holds = (A == 64) || (lane < A);
    const float decay_p = lr * lp, decay_q = lr * lq;

    int64_t c_batch = worker, n_batch = worker;
    int c_off = 0, n_off = 0;
    auto advance = [&](int64_t& b, int& o) {
        o += 64;
        if (o >= f) {
            o = 0;
            b += W;
        }
    };
    auto load_chunk = [&](int64_t b, int o, int& cu, int& cv, float& cr, int& cnt) {
        const int64_t s0 = b * (int64_t)f + o;
        const int64_t rem = nnz - s0;
        cnt = rem <= 0 ? 0 : (rem >= 64 ? 64 : (int)rem);
        const int64_t i = s0 + (lane < cnt ? lane : 0);
        const Sample* sp = S + (cnt > 0 ? i : 0);
        cu = __builtin_nontemporal_load(&sp->u);
        cv = __builtin_nontemporal_load(&sp->v);
        cr = __builtin_nontemporal_load(&sp->r);
    };

    if (nnz <= 0 || worker * (int64_t)f >= nnz)
        return;
    int cU, cV, nU, nV, ccnt, ncnt;
    float cR, nR;
    load_chunk(c_batch, c_off, cU, cV, cR, ccnt);
    advance(n_batch, n_off);
    load_chunk(n_batch, n_off, nU, nV, nR, ncnt);

    WorkerState<KP, T, D> st;
    typedef typename WorkerState<KP, T, D>::V V;
#pragma unroll
    for (int d = 0; d < D; ++d) {
        st.su[d] = st.sv[d] = st.hu[d] = st.hv[d] = -1;
        st.sr[d] = 0.f;
        st.sp[d] = st.sq[d] = st.hp[d] = st.hq[d] = V{};
        st.cp[d] = st.cq[d] = false;
    }

    // request the rows of the sample at lane `xl` of a chunk's metadata
    auto issue = [&](int slot, int mu, int mv, float mr, int xl, int cnt) {
        const bool ok = xl < cnt;
        const int u = __builtin_amdgcn_readlane(mu, xl);
        const int v = __builtin_amdgcn_readlane(mv, xl);
        const float r = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(mr), xl));
        st.su[slot] = ok ? u : -1;
        st.sv[slot] = ok ? v : -1;
        st.sr[slot] = r;
        if constexpr (ATOM) {
            // rows updated with atomic adds: every row, or the hot ones
            st.cp[slot] = coh.hot_p == nullptr || hot_bit(coh.hot_p, ok ? u : 0);
            st.cq[slot] = coh.hot_q == nullptr || hot_bit(coh.hot_q, ok ? v : 0);
        }
        if constexpr (ATOM && COH == kCohBoth) {
            st.sp[slot] = ld_coh(reinterpret_cast<const V*>(P + (int64_t)(ok ? u : 0) * KP + col));
            st.sq[slot] = ld_coh(reinterpret_cast<const V*>(Q + (int64_t)(ok ? v : 0) * KP + col));
        } else if constexpr (COH != kCohOff) {
            const bool cp = coh.p && !hot_bit(coh.hot_p, ok ? u : 0);
            const bool cq = coh.q && !hot_bit(coh.hot_q, ok ? v : 0);
            st.cp[slot] = cp;
            st.cq[slot] = cq;
            const V* pr = reinterpret_cast<const V*>(P + (int64_t)(ok ? u : 0) * KP + col);
            const V* qr = reinterpret_cast<const V*>(Q + (int64_t)(ok ? v : 0) * KP + col);
            if constexpr (COH == kCohBoth) {
                st.sp[slot] = cp ? ld_coh(pr) : *pr;
                st.sq[slot] = cq ? ld_coh(qr) : *qr;
            } else {
                st.sp[slot] = *pr;
                st.sq[slot] = *qr;
            }
        } else if constexpr (BUF) {
            st.sp[slot] = bp.template ld<V>(cb, (uint32_t)(ok ? u : 0) * kRowBytes);
            st.sq[slot] = bq.template ld<V>(cb, (uint32_t)(ok ? v : 0) * kRowBytes);
        } else {
            st.sp[slot] = R::ld(P + (int64_t)(ok ? u : 0) * KP + col);
            st.sq[slot] = R::ld(Q + (int64_t)(ok ? v : 0) * KP + col);
        }
    };

    // update the sample in slot j
    auto process = [&](int j, int64_t pos) {
        const int u = st.su[j], v = st.sv[j];
        // a row that one of the previous D-1 samples rewrote is taken from that
        // sample's stored value (whole vectors; the nearest writer wins)
        V pv = st.sp[j], qv = st.sq[j];
        // Wave-uniform test: where rows rarely repeat within D samples a
        // scalar branch skips the selects; the hot-row variant (SKIP), whose
        // rows repeat nearly every sample, always selects.  So do lanes
        // holding more than 16 bytes of a row (binary32 at KP = 512): the
        // branched form of those produced wrong values at depths 2 and 4 in
        // this compiler (caught by the single-worker parity tests), the
        // always-select form is exact.
        constexpr bool kAlways = SKIP || sizeof(V) > 16;
        bool fwd = kAlways;
#pragma unroll
        for (int d = 1; d < D && !kAlways; ++d) {
            const int h = (j - d + D) % D;
            fwd |= (st.hu[h] == u) | (st.hv[h] == v);
        }
        if (__builtin_expect(fwd, 0)) {
#pragma unroll
            for (int d = D - 1; d >= 1; --d) {
                const int h = (j - d + D) % D;
                pv = pick(st.hu[h] == u, st.hp[h], pv);
                qv = pick(st.hv[h] == v, st.hq[h], qv);
            }
        }
        float p[E], q[E];
        R::widen(pv, p);
        R::widen(qv, q);
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e)
            dot += p[e] * q[e];
        if constexpr (A < 64)
            dot = holds ? dot : 0.f; // idle lanes hold a copy of column 0
        dot = wave_sum(dot);
        const float err = st.sr[j] - dot;
        if constexpr (ATOM) {
            // the changes lr (err q - lp p) and lr (err p - lq q), both from
            // the values before the step, added atomically to the rows marked
            // for it and stored (value plus change) to the others; with one
            // sample in flight the next load of this wavefront is issued after
            // these writes and sees them
            float dp[E], dq[E];
#pragma unroll
            for (int e = 0; e < E; ++e) {
                dp[e] = lr * (err * q[e] - lp * p[e]);
                dq[e] = lr * (err * p[e] - lq * q[e]);
            }
            if (holds) {
                T* pr = P + (int64_t)u * KP + col;
                T* qr = Q + (int64_t)v * KP + col;
                if (st.cp[j]) {
                    if constexpr (sizeof(T) == 4 && A == 64 && (E == 2 || E == 4))
                        add_row_t<T, E>(P + (int64_t)u * KP, lane, dp);
                    else
                        add_row<T, E>(pr, dp);
                } else {
#pragma unroll
                    for (int e = 0; e < E; ++e)
                        dp[e] += p[e];
                    R::store(pr, dp);
                }
                if (st.cq[j]) {
                    if constexpr (sizeof(T) == 4 && A == 64 && (E == 2 || E == 4))
                        add_row_t<T, E>(Q + (int64_t)v * KP, lane, dq);
                    else
                        add_row<T, E>(qr, dq);
                } else {
#pragma unroll
                    for (int e = 0; e < E; ++e)
                        dq[e] += q[e];
                    R::store(qr, dq);
                }
            }
            if constexpr (DBG) {
                if (dbg.visits && lane == 0) {
                    const int64_t idx = dbg.orig ? dbg.orig[pos] : pos;
                    atomicAdd(dbg.visits + idx, 1u);
                }
            }
            return;
        }
        if constexpr (sizeof(T) == 2) {
            // Binary16 storage (instruction-issue bound): p + lr (err q - lp p)
            // evaluated as (p + (lr err) q) - (lr lp) p, two fused operations
            // per element, both from the values before the step, which read the
            // stored halves directly (mixed-precision fmas, no conversions).
            // Folding the decay into one factor 1 - lr lp instead would round
            // that factor once for every update, a bias that builds up on rows
            // updated millions of times.
            const float step = lr * err;
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const float pe = p[e], qe = q[e];
                p[e] = __builtin_fmaf(-decay_p, pe, __builtin_fmaf(step, qe, pe));
                q[e] = __builtin_fmaf(-decay_q, qe, __builtin_fmaf(step, pe, qe));
            }
        } else {
            // Binary32 storage (memory bound): the update as written; the
            // shorter form above moves this kernel's memory waits (measured
            // 13 % slower on the Yahoo shape).
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const float pe = p[e], qe = q[e];
                p[e] = pe + lr * (err * qe - lp * pe);
                q[e] = qe + lr * (err * pe - lq * qe);
            }
        }
        const V np = R::narrow(p), nq = R::narrow(q);
        // SKIP: a row that one of the next D-1 samples (already issued, so
        // certain to be processed) updates again takes its value from this
        // one by forwarding and stores it later, so this store goes to the
        // wavefront's private sink rows instead (a select, not a branch, so
        // the memory-counter waits stay static).  Hot rows then see one store per
        // run of in-flight updates, and the worker's final values are
        // unchanged.  This pays where many workers share one L2 and its hot
        // lines (block-scheduled epochs).
        T* pbase = P + (int64_t)u * KP;
        T* qbase = Q + (int64_t)v * KP;
        if constexpr (SKIP) {
            bool p_again = false, q_again = false;
#pragma unroll
            for (int d = 1; d < D; ++d) {
                const int h = (j + d) % D;
                p_again |= st.su[h] == u;
                q_again |= st.sv[h] == v;
            }
            pbase = p_again ? sink : pbase;
            qbase = q_again ? sink + KP : qbase;
        }
        if (holds) {
            if constexpr (COH != kCohOff) {
                V* pr = reinterpret_cast<V*>(pbase + col);
                V* qr = reinterpret_cast<V*>(qbase + col);
                if (st.cp[j])
                    st_coh<COH>(pr, np);
                else
                    *pr = np;
                if (st.cq[j])
                    st_coh<COH>(qr, nq);
                else
                    *qr = nq;
            } else if constexpr (BUF) {
                bp.template st<V>(np, cb, (uint32_t)u * kRowBytes);
                bq.template st<V>(nq, cb, (uint32_t)v * kRowBytes);
            } else {
                R::st(pbase + col, np);
                R::st(qbase + col, nq);
            }
        }
        st.hu[j] = u;
        st.hv[j] = v;
        st.hp[j] = np;
        st.hq[j] = nq;
        if constexpr (DBG) {
            if (dbg.visits && lane == 0) {
                const int64_t idx = dbg.orig ? dbg.orig[pos] : pos;
                atomicAdd(dbg.visits + idx, 1u);
            }
        }
    };

    int batches = 0;
    // prologue: positions 0 .. D-2 of the first chunk
#pragma unroll
    for (int d = 0; d < D - 1; ++d)
        issue(d, cU, cV, cR, d, ccnt);

    // One chunk of 64 positions; metadata of this chunk in (aU, aV, aR, acnt),
    // of the next in (bU, bV, bR, bcnt).  The registers of a finished chunk
    // receive the chunk after next, so the two sets alternate without copies.
    auto chunk = [&](int& aU, int& aV, float& aR, int& acnt, int bU, int bV, float bR, int bcnt) -> bool {
        const int64_t cbase = c_batch * (int64_t)f + c_off;
        if constexpr (DBG) {
            if (dbg.trace && c_off == 0 && lane == 0)
                dbg.trace[c_batch] = (int32_t)worker;
        }
        if (sync.every > 0 && c_off == 0 && ++batches % sync.every == 0) {
            if (sync.leader) {
                release_agent();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            } else if (sync.l1) {
                asm volatile("buffer_inv sc0" ::: "memory");
            }
        }
        for (int g = 0; g < 64 - D; g += D) { // look-ahead stays inside this chunk
#pragma unroll
            for (int j = 0; j < D; ++j) {
                const int x = g + j;
                if (x >= acnt)
                    return false;
                issue((j + D - 1) % D, aU, aV, aR, x + D - 1, acnt);
                process(j, cbase + x);
            }
        }
#pragma unroll
        for (int j = 0; j < D; ++j) { // last group: look-ahead reaches into the next chunk
            const int x = 64 - D + j;
            if (x >= acnt)
                return false;
            if (j == 0)
                issue((j + D - 1) % D, aU, aV, aR, 63, acnt);
            else
                issue((j + D - 1) % D, bU, bV, bR, j - 1, bcnt);
            process(j, cbase + x);
        }
        if (bcnt == 0)
            return false;
        c_batch = n_batch;
        c_off = n_off;
        advance(n_batch, n_off);
        load_chunk(n_batch, n_off, aU, aV, aR, acnt);
        return true;
    };
    for (;;) {
        if (!chunk(cU, cV, cR, ccnt, nU, nV, nR, ncnt))
            return;
        if (!chunk(nU, nV, nR, ncnt, cU, cV, cR, ccnt))
            return;
    }
}

// ---------------------------------------------------------------------------
// Two batch-Hogwild! workers per wavefront.  At KP = 32 a one-worker
// wavefront would leave half of its lanes idle; at wider rows each lane of a
// half holds KP/32 values (at most 16 bytes), so one memory instruction moves
// the rows of two samples.
//
// Lanes 0-31 are worker 2 h and lanes 32-63 worker 2 h + 1 of the W workers
// (h = the wavefront's index); each half holds a row across its 32 lanes and
// runs the sequence of run_worker's worker (batches b = worker, worker+W, ...
// of f consecutive samples, in array order) with the same in-flight window,
// forwarding and arithmetic.  The two halves step through their sequences
// together: batch b of lanes 0-31 goes with batch b + 1 of lanes 32-63 at the
// same offset, so the chunk offset is common and only the sample counts
// differ (the second half's count never exceeds the first's, its samples lying
// f further on).  A position past a half's count loads row 0 and stores
// nothing.  Each half's dot product is a 32-lane sum; with one active half it
// adds the same terms in the same order as run_worker's 64-lane sum (whose
// idle lanes add zeros) at KP = 32, so a lone worker computes the same bits
// either way there; wider rows sum their products in another order.
// ---------------------------------------------------------------------------
//
// SKIP (block-scheduled epochs at rows wider than 32 values): as in
// run_worker, a row that one of the half's next D-1 samples updates again is
// stored to the half's private sink row instead (sink: 4 rows per wavefront,
// P and Q of lanes 0-31, then of lanes 32-63).
template <int KP, typename T, int D, bool DBG, bool BUF = false, bool SKIP = false>
__device__ __forceinline__ void run_worker_half(const Sample* __restrict__ S, int64_t nnz, int64_t W, int64_t wave,
                                                int f, T* __restrict__ P, T* __restrict__ Q, float lr, float lp,
                                                float lq, const DebugSink dbg,
                                                const CacheSync sync = CacheSync{0, false, false},
                                                T* __restrict__ sink = nullptr)
{
    constexpr int H = 32;      // positions per chunk and half; lanes per half
    constexpr int E = KP / H;  // values per lane
    typedef Row<T, E> R;
    typedef typename VecT<T, E>::type V;
    static_assert(KP % H == 0 && sizeof(V) <= 16, "rows of 32 to 512 values, at most 16 bytes per lane");
    static_assert(!BUF || sizeof(V) == 4, "buffer rows: one dword per lane");
    static_assert(!(BUF && SKIP), "buffer rows: no store redirection");
    static_assert(H % D == 0 && D <= 16, "depth must divide 32");

    const int lane = lane_id();
    const bool hi = lane >= H;           // lanes 32-63
    const int hl = lane & (H - 1);        // lane within the half
    const int col = hl * E;               // first value of a row held by this lane
    const int64_t w0 = 2 * wave;          // worker of lanes 0-31
    const bool two = w0 + 1 < W;          // lanes 32-63 are a worker too
    const Buf bp(P), bq(Q);
    const uint32_t cb = (uint32_t)(col * sizeof(T));
    constexpr uint32_t kRowBytes = (uint32_t)(KP * sizeof(T));
    const float decay_p = lr * lp, decay_q = lr * lq;

    // batch of lanes 0-31 (lanes 32-63 work on the next one) and common offset
    int64_t c_batch = w0, n_batch = w0;
    int c_off = 0, n_off = 0;
    auto advance = [&](int64_t& b, int& o) {
        o += H;
        if (o >= f) {
            o = 0;
            b += W;
        }
    };
    auto count = [&](int64_t s0) -> int {
        const int64_t rem = nnz - s0;
        return rem <= 0 ? 0 : (rem >= H ? H : (int)rem);
    };
    // metadata of one chunk: lane i of each half holds that half's sample i
    auto load_chunk = [&](int64_t b, int o, int& cu, int& cv, float& cr, int& c0, int& c1) {
        const int64_t s0 = b * (int64_t)f + o;
        c0 = count(s0);
        c1 = two ? count(s0 + f) : 0;
        const int mine = hi ? c1 : c0;
        const int64_t i = s0 + (hi ? f : 0) + (hl < mine ? hl : 0);
        const Sample* sp = S + (mine > 0 ? i : 0);
        cu = __builtin_nontemporal_load(&sp->u);
        cv = __builtin_nontemporal_load(&sp->v);
        cr = __builtin_nontemporal_load(&sp->r);
    };

    if (nnz <= 0 || w0 >= W || w0 * (int64_t)f >= nnz)
        return;
    int cU, cV, nU, nV, c0, c1, n0, n1;
    float cR, nR;
    load_chunk(c_batch, c_off, cU, cV, cR, c0, c1);
    advance(n_batch, n_off);
    load_chunk(n_batch, n_off, nU, nV, nR, n0, n1);

    int su[D], sv[D], hu[D], hv[D];
    float sr[D];
    V sp[D], sq[D], hp[D], hq[D];
#pragma unroll
    for (int d = 0; d < D; ++d) {
        su[d] = sv[d] = hu[d] = hv[d] = -1;
        sr[d] = 0.f;
        sp[d] = sq[d] = hp[d] = hq[d] = V{};
    }

    // request the rows of each half's sample at position xl of a chunk.  Lane
    // xl of each half holds it; one backward permute per field hands it to
    // every lane of that half (the loop bounds are wave-uniform, so all 64
    // lanes are active here), in place of two lane reads and a select.
    const int src_half = hi ? 4 * H : 0; // byte address of lane 32
    auto issue = [&](int slot, int mu, int mv, float mr, int xl, int k0, int k1) {
        const bool ok = xl < (hi ? k1 : k0);
        const int src = src_half + 4 * xl;
        const int u = __builtin_amdgcn_ds_bpermute(src, mu);
        const int v = __builtin_amdgcn_ds_bpermute(src, mv);
        su[slot] = ok ? u : -1;
        sv[slot] = ok ? v : -1;
        sr[slot] = __int_as_float(__builtin_amdgcn_ds_bpermute(src, __float_as_int(mr)));
        if constexpr (BUF) {
            sp[slot] = bp.template ld<V>(cb + (uint32_t)(ok ? u : 0) * kRowBytes, 0);
            sq[slot] = bq.template ld<V>(cb + (uint32_t)(ok ? v : 0) * kRowBytes, 0);
        } else {
            sp[slot] = R::ld(P + (int64_t)(ok ? u : 0) * KP + col);
            sq[slot] = R::ld(Q + (int64_t)(ok ? v : 0) * KP + col);
        }
    };

    // update each half's sample in slot j (pos: position of the first half's
    // sample in S; the second half's is f further)
    auto process = [&](int j, int64_t pos) {
        const int u = su[j], v = sv[j];
        V pv = sp[j], qv = sq[j];
        bool fwd = false;
#pragma unroll
        for (int d = 1; d < D; ++d) {
            const int h = (j - d + D) % D;
            fwd |= (hu[h] == u) | (hv[h] == v);
        }
        if (__builtin_expect(__builtin_amdgcn_ballot_w64(fwd) != 0, 0)) {
#pragma unroll
            for (int d = D - 1; d >= 1; --d) {
                const int h = (j - d + D) % D;
                pv = pick(hu[h] == u, hp[h], pv);
                qv = pick(hv[h] == v, hq[h], qv);
            }
        }
        float p[E], q[E];
        R::widen(pv, p);
        R::widen(qv, q);
        float dot = 0.f;
#pragma unroll
        for (int e = 0; e < E; ++e)
            dot += p[e] * q[e];
        // the lane's sum is rounded before the cross-lane sum (the empty asm
        // keeps it from fusing into the first cross-lane add), as in run_worker
        asm volatile("" : "+v"(dot));
        const float err = sr[j] - half_sum(dot);
        if constexpr (sizeof(T) == 2) {
            const float step = lr * err;
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const float pe = p[e], qe = q[e];
                p[e] = __builtin_fmaf(-decay_p, pe, __builtin_fmaf(step, qe, pe));
                q[e] = __builtin_fmaf(-decay_q, qe, __builtin_fmaf(step, pe, qe));
            }
        } else {
#pragma unroll
            for (int e = 0; e < E; ++e) {
                const float pe = p[e], qe = q[e];
                p[e] = pe + lr * (err * qe - lp * pe);
                q[e] = qe + lr * (err * pe - lq * qe);
            }
        }
        const V np = R::narrow(p), nq = R::narrow(q);
        if (u >= 0) {
            if constexpr (BUF) {
                bp.template st<V>(np, cb + (uint32_t)u * kRowBytes, 0);
                bq.template st<V>(nq, cb + (uint32_t)v * kRowBytes, 0);
            } else if constexpr (SKIP) {
                // the half's next D-1 samples (issued, so processed before
                // this half stops) take a row they update again from this one
                // by forwarding
                bool p_again = false, q_again = false;
#pragma unroll
                for (int d = 1; d < D; ++d) {
                    const int h = (j + d) % D;
                    p_again |= su[h] == u;
                    q_again |= sv[h] == v;
                }
                R::st(p_again ? sink + (hi ? 2 * KP : 0) + col : P + (int64_t)u * KP + col, np);
                R::st(q_again ? sink + (hi ? 3 * KP : KP) + col : Q + (int64_t)v * KP + col, nq);
            } else {
                R::st(P + (int64_t)u * KP + col, np);
                R::st(Q + (int64_t)v * KP + col, nq);
            }
        }
        hu[j] = u;
        hv[j] = v;
        hp[j] = np;
        hq[j] = nq;
        if constexpr (DBG) {
            if (dbg.visits && hl == 0 && u >= 0) {
                const int64_t at = pos + (hi ? f : 0);
                atomicAdd(dbg.visits + (dbg.orig ? dbg.orig[at] : at), 1u);
            }
        }
    };

    int batches = 0;
#pragma unroll
    for (int d = 0; d < D - 1; ++d)
        issue(d, cU, cV, cR, d, c0, c1);

    // one chunk of H positions per half: metadata of this chunk in (aU, aV,
    // aR; counts a0, a1), of the next in (bU, bV, bR; b0, b1); the registers of
    // a finished chunk receive the chunk after next
    auto chunk = [&](int& aU, int& aV, float& aR, int& a0, int& a1, int bU, int bV, float bR, int b0,
                     int b1) -> bool {
        const int64_t cbase = c_batch * (int64_t)f + c_off;
        if constexpr (DBG) {
            if (dbg.trace && c_off == 0 && hl == 0 && (hi ? a1 : a0) > 0)
                dbg.trace[c_batch + (hi ? 1 : 0)] = (int32_t)(w0 + (hi ? 1 : 0));
        }
        if (sync.every > 0 && c_off == 0 && ++batches % sync.every == 0) {
            if (sync.leader) {
                release_agent();
                __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            } else if (sync.l1) {
                asm volatile("buffer_inv sc0" ::: "memory");
            }
        }
        for (int g = 0; g < H - D; g += D) { // look-ahead stays inside this chunk
#pragma unroll
            for (int j = 0; j < D; ++j) {
                const int x = g + j;
                if (x >= a0)
                    return false;
                issue((j + D - 1) % D, aU, aV, aR, x + D - 1, a0, a1);
                process(j, cbase + x);
            }
        }
#pragma unroll
        for (int j = 0; j < D; ++j) { // last group: look-ahead reaches into the next chunk
            const int x = H - D + j;
            if (x >= a0)
                return false;
            if (j == 0)
                issue((j + D - 1) % D, aU, aV, aR, H - 1, a0, a1);
            else
                issue((j + D - 1) % D, bU, bV, bR, j - 1, b0, b1);
            process(j, cbase + x);
        }
        if (b0 == 0)
            return false;
        c_batch = n_batch;
        c_off = n_off;
        advance(n_batch, n_off);
        load_chunk(n_batch, n_off, aU, aV, aR, a0, a1);
        return true;
    };
    for (;;) {
        if (!chunk(cU, cV, cR, c0, c1, nU, nV, nR, n0, n1))
            return;
        if (!chunk(nU, nV, nR, n0, n1, cU, cV, cR, c0, c1))
            return;
    }
}

} // namespace mfsgd
