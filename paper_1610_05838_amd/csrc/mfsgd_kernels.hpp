// mfsgd_kernels.hpp -- the gfx950 kernels and their launchers, instantiated
// once per storage type (mfsgd_kernels_f32.hip, mfsgd_kernels_f16.hip).
#pragma once

#include "mfsgd_device.hpp"
#include "mfsgd_launch.hpp"

namespace mfsgd {

constexpr int kHogwildBlock = 256; // 4 wavefronts per workgroup, each an independent worker

// batch-Hogwild! over the whole GPU in one address space (section 3.2.2):
// wavefront w of the grid is worker w.  The XCDs' L2 caches are not coherent
// with each other, so rows that several XCDs touch are updated in per-XCD
// copies until evicted; the block-scheduled kernel below is the coherent form.
template <int KP, typename T, int D, bool DBG, bool BUF = false, int COH = kCohOff, bool ATOM = false>
__global__ __launch_bounds__(kHogwildBlock) void k_hogwild(const Sample* __restrict__ S, int64_t nnz, int64_t W,
                                                           int f, T* __restrict__ P, T* __restrict__ Q, float lr,
                                                           float lp, float lq, DebugSink dbg, int sync_every,
                                                           int sync_l1, int nx, Coherence coh)
{
    const int64_t worker = uniform64((int64_t)blockIdx.x * (kHogwildBlock / 64) + (threadIdx.x >> 6));
    if (worker >= W)
        return;
    // workgroups are dealt to XCDs round-robin: the first wavefront of each of
    // the first nx workgroups leads its XCD's cache flushes
    const CacheSync sync{sync_every, (int)blockIdx.x < nx && (threadIdx.x >> 6) == 0, sync_l1 != 0};
    run_worker<KP, T, D, DBG, false, BUF, COH, ATOM>(S, nnz, W, worker, f, P, Q, lr, lp, lq, dbg, sync, nullptr, coh);
}

// Row widths whose half-wavefront layout holds at most 16 bytes per lane.
template <int KP, typename T>
constexpr bool kHalfRows = sizeof(T) * KP <= 16 * 32;

// The same with two workers per wavefront (run_worker_half), wavefront h of
// the grid being workers 2 h and 2 h + 1.
template <int KP, typename T, int D, bool DBG, bool BUF = false>
__global__ __launch_bounds__(kHogwildBlock) void k_hogwild_half(const Sample* __restrict__ S, int64_t nnz, int64_t W,
                                                                int f, T* __restrict__ P, T* __restrict__ Q, float lr,
                                                                float lp, float lq, DebugSink dbg, int sync_every,
                                                                int sync_l1, int nx)
{
    const int64_t wave = uniform64((int64_t)blockIdx.x * (kHogwildBlock / 64) + (threadIdx.x >> 6));
    if (2 * wave >= W)
        return;
    const CacheSync sync{sync_every, (int)blockIdx.x < nx && (threadIdx.x >> 6) == 0, sync_l1 != 0};
    run_worker_half<KP, T, D, DBG, BUF>(S, nnz, W, wave, f, P, Q, lr, lp, lq, dbg, sync);
}

// Block-scheduled epoch: wavefront-update (section 3.2.3), and
// batch-Hogwild! partitioned over the GPU's coherence domains.
//
// The s x s grid of blocks is processed in s waves.  Team (row block) t in
// wave w works on column block sigma_t(w) = C[(t + O[w]) mod s], so the blocks
// of one wave share no row and no column.  A column ticket counts the waves
// completed on its column: block (t, w) opens once ticket[sigma_t(w)] has
// reached w, and the wavefront that finishes the block's last batch sets it to
// w + 1 (each column is used by exactly one team per wave).
//
// Inside an open block the batches of f consecutive samples are claimed one
// at a time from the block's claim counter, and each is run serially by one
// wavefront (run_worker); concurrent batches of a block race as in
// batch-Hogwild!.  A team's teams-mates may already work on the team's next
// block while the last batches of the previous one run (the two share only
// the team's row block).  cursor[t] is the lowest wave of team t that may still
// have unclaimed batches.
//
// Every team lives on one XCD (pooled teams: a workgroup reads its XCD from
// the hardware and joins a team placed there; one-wavefront teams are single
// wavefronts), so all updates of a team meet in that XCD's L2.  In pool mode a
// wavefront serves its home team first and otherwise any open block of the
// other teams on its XCD; without pool mode (one-wavefront teams: the
// deterministic schedule) only its home team.  Rows move between XCDs only
// at block hand-over: the releasing wavefront writes its XCD's L2 back
// (agent-scope release) before it advances the ticket, and a wavefront
// entering a block invalidates its caches (agent-scope acquire) first.
//
// With free_run, blocks open without their ticket (batch-Hogwild!
// partitioned over the XCDs without waiting): teams still walk their columns
// in wavefront order, but a team that is ahead may share a column block with
// one that lags, and that block's rows are then updated on two XCDs at once.
//
// Nothing waits for a particular workgroup: work is claimed, not assigned,
// so workgroups that become resident late (or never, before the others
// finish) are harmless, and the grid may be as large as the occupancy allows.
// A wait for an open block that exceeds spin_limit polls raises *err; every
// wavefront that then finds nothing to claim leaves, so the grid drains.
//
// Claims are counted in units of 64 samples: a block's first units go in
// head claims of f samples (2 f with HALF), its last `tail` units one at a
// time, so that the block ends with many wavefronts finishing small pieces.
// Among the open blocks a wavefront can serve, it takes the one with the
// largest critical-path weight prio[t*s + w] (the work that must still
// follow the block one step at a time: the team's later blocks and the
// column's, k_block_priority), the first in its preference order (home team
// first) among equals or when prio is null.
//
// sched: [0, G2) units finished per (team, wave), [G2, 2 G2) head claims
// taken per (team, wave), [2 G2, 2 G2 + kMaxGrid) cursor per team, one event
// counter, kMaxGrid workgroups arrived per XCD, then [.., + G2) unit claims
// taken per (team, wave), where G2 = kMaxGrid^2; all zero at launch.
//
// Debug (trace != nullptr): trace[t*s + w] = column of team t in wave w, and
// after those s*s entries two stamps per (team, wave) from the event counter:
// the earliest claim of any of the block's batches and the completion of its
// last batch (taken before the column's ticket moves on).  In every column,
// the block of wave w+1 must be claimed only after the block of wave w was
// completed; the host checks that from the stamps.
//
// HALF (rows of at most 16 bytes per half-wavefront lane): a wavefront claims
// two consecutive batches of the block at once and runs them as two workers,
// one per half (run_worker_half); the block's finished count advances by the
// batches run.  At KP = 32 this replaces skipped stores; at wider rows SKIP
// applies per half.

template <int KP, typename T, int D, bool DBG, bool SKIP, bool HALF = false, bool ATOM = false>
__global__ __launch_bounds__(256) void k_blocked(const Sample* __restrict__ Sp, const int64_t* __restrict__ bstart,
                                                 int s, int xslots, const int32_t* __restrict__ tmap,
                                                 const int32_t* __restrict__ xteams, int nx, int pool,
                                                 const uint32_t* __restrict__ prio_tw, int free_run,
                                                 uint64_t sigma_c, uint64_t sigma_o, uint32_t tail, T* __restrict__ P,
                                                 T* __restrict__ Q, float lr, float lp, float lq, int f,
                                                 uint32_t* tickets, uint32_t* sched, uint32_t spin_limit, int* err,
                                                 DebugSink dbg, int32_t* trace, T* __restrict__ sink,
                                                 Coherence coh)
{
    static_assert(!HALF || (KP == 32 ? !SKIP : kHalfRows<KP, T>),
                  "half-wavefront workers: at most 16 bytes of a row per lane; at 32 values no store redirection");
    constexpr uint32_t kClaim = HALF ? 2u : 1u; // batches per head claim
    constexpr uint32_t kUnit = 64;              // samples per claim unit
    __shared__ int Cperm[kMaxGrid], Ooff[kMaxGrid];
    __shared__ int s_tm, s_x;
    uint32_t* const arrived = sched + 2 * kMaxGrid * kMaxGrid + kMaxGrid + 1;
    if (threadIdx.x == 0) {
        if (xslots > 0) {
            // pooled teams: the XCD this workgroup runs on (hardware register)
            // and its arrival order there select its team, so a team's
            // wavefronts share one L2 whatever order the dispatcher uses
            unsigned xcc;
            asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(xcc));
            const int x = (int)(xcc & 0xfu) % nx;
            const uint32_t slot =
                __hip_atomic_fetch_add(arrived + x, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            s_x = x;
            s_tm = slot < (uint32_t)xslots ? tmap[(int64_t)x * xslots + slot] : -1;
        } else {
            s_x = 0;
            s_tm = tmap[blockIdx.x];
        }
        shuffle_perm(sigma_c, s, Cperm);
        shuffle_perm(sigma_o, s, Ooff);
    }
    __syncthreads();
    const int tm = s_tm;
    if (tm < 0)
        return;
    const int home = tm >> 16;
    const int lane = lane_id();
    const int waves = blockDim.x >> 6;
    const int wv = uniform(threadIdx.x >> 6);
    uint32_t* const fin = sched;
    uint32_t* const claim = sched + kMaxGrid * kMaxGrid;
    uint32_t* const cursor = sched + 2 * kMaxGrid * kMaxGrid;
    uint32_t* const events = cursor + kMaxGrid;
    uint32_t* const claim2 = events + 1 + kMaxGrid; // after the arrival counters
    uint32_t* const stamps = trace ? reinterpret_cast<uint32_t*>(trace) + (int64_t)s * s : nullptr;
    // after the event stamps: the same two moments on the 100 MHz realtime clock (low 32 bits)
    uint32_t* const clocks = trace ? stamps + 2 * (int64_t)s * s : nullptr;
    // private rows per wavefront of the grid for skipped stores: P and Q (of
    // each half with HALF); the grid's sink holds four per wavefront
    T* const my_sink = SKIP ? sink + ((int64_t)blockIdx.x * waves + wv) * (HALF ? 4 : 2) * KP : nullptr;

    // lane j < nt watches the j-th team of this wavefront's preference order:
    // the home team, then the other teams of the XCD in list order
    const int32_t* xt = xteams + (int64_t)s_x * (kMaxGrid + 1);
    const int nt = pool ? xt[0] : 1;
    int hidx = 0;
    for (int j = 0; pool && j < nt; ++j)
        hidx = xt[1 + j] == home ? j : hidx;
    const int lt = lane < nt ? (pool ? xt[1 + (hidx + lane) % nt] : home) : -1;

    int64_t entered = -1; // (team, wave) whose data this wavefront has acquired
    uint32_t polls = 0;
    for (;;) {
        int cw = s;
        bool open = false;
        uint32_t prio = 0;
        if (lt >= 0) {
            cw = (int)__hip_atomic_load(cursor + lt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (cw < s) {
                const int col = Cperm[(lt + Ooff[cw]) % s];
                open = free_run ||
                       __hip_atomic_load(tickets + col, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >= (uint32_t)cw;
                prio = prio_tw ? prio_tw[(int64_t)lt * s + cw] : 0u;
            }
        }
        if (__builtin_amdgcn_ballot_w64(cw < s) == 0)
            return; // every batch of every watched team has been claimed
        const uint64_t avail = __builtin_amdgcn_ballot_w64(open);
        if (avail == 0) {
            int stop = 0;
            if (lane == 0)
                stop = ++polls > spin_limit || __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (__builtin_amdgcn_readfirstlane(stop)) {
                if (lane == 0)
                    __hip_atomic_fetch_or(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                return;
            }
            __builtin_amdgcn_s_sleep(4);
            continue;
        }
        polls = 0;
        // the open block with the longest chain behind it, the first in
        // preference order (home team first) among equals
        int j = (int)__builtin_ctzll(avail);
        if (prio_tw) {
            uint32_t best = __builtin_amdgcn_readlane(prio, j);
            for (uint64_t rest = avail & (avail - 1); rest; rest &= rest - 1) {
                const int l = (int)__builtin_ctzll(rest);
                const uint32_t p = __builtin_amdgcn_readlane(prio, l);
                if (p > best) {
                    best = p;
                    j = l;
                }
            }
        }
        const int t = __builtin_amdgcn_readlane(lt, j);
        const int w = __builtin_amdgcn_readlane(cw, j);
        const int col = Cperm[(t + Ooff[w]) % s];
        const int64_t tw = (int64_t)t * s + w;
        const int64_t b = (int64_t)t * s + col;
        const int64_t lo = bstart[b], hi = bstart[b + 1];
        // Claims are counted in units of kUnit samples: head claims of f
        // samples (two batches with HALF) from counter A while the block has
        // more than `tail` units left unclaimed, then single units from
        // counter B, so the block's last work is spread over many wavefronts
        // in small pieces instead of a few whole batches.
        const uint32_t nu = (uint32_t)((hi - lo + kUnit - 1) / kUnit);
        const uint32_t big = kClaim * (uint32_t)f / kUnit;
        const uint32_t split = tail > 0 ? (nu > tail ? (nu - tail) / big * big : 0u) : nu;
        const uint32_t heads = (split + big - 1) / big;
        uint32_t idx = 0, take = 0, got = 0;
        if (lane == 0) {
            const uint32_t a = __hip_atomic_fetch_add(claim + tw, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (a < heads) {
                idx = a * big;
                take = split - idx < big ? split - idx : big;
            } else {
                const uint32_t k = __hip_atomic_fetch_add(claim2 + tw, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                idx = split + k;
                take = idx < nu ? 1u : 0u;
                got = k; // 0 for the first claimant of an exhausted block
            }
        }
        idx = __builtin_amdgcn_readfirstlane(idx);
        take = __builtin_amdgcn_readfirstlane(take);
        got = __builtin_amdgcn_readfirstlane(got);
        if (take == 0) {
            // nothing left to claim in this block: move the team's cursor on;
            // an empty block is released by its only claimant
            if (lane == 0) {
                if (nu == 0 && got == 0) {
                    if (trace) {
                        trace[tw] = col;
                        const uint32_t e =
                            __hip_atomic_fetch_add(events, 2u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        stamps[2 * tw] = e;
                        stamps[2 * tw + 1] = e + 1u;
                        const uint32_t now = (uint32_t)__builtin_amdgcn_s_memrealtime();
                        clocks[2 * tw] = now;
                        clocks[2 * tw + 1] = now;
                        __builtin_amdgcn_s_waitcnt(0);
                    }
                    release_agent();
                    __hip_atomic_store(tickets + col, (uint32_t)(w + 1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                }
                uint32_t expect = (uint32_t)w;
                __hip_atomic_compare_exchange_strong(cursor + t, &expect, (uint32_t)(w + 1), __ATOMIC_RELAXED,
                                                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            continue;
        }
        if (trace && lane == 0) {
            if (idx == 0)
                trace[tw] = col;
            const uint32_t e = __hip_atomic_fetch_add(events, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_fetch_min(stamps + 2 * tw, e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            if (idx == 0)
                clocks[2 * tw] = (uint32_t)__builtin_amdgcn_s_memrealtime();
            __builtin_amdgcn_s_waitcnt(0); // stamped before any of the batch's rows is read
        }
        if (entered != tw) {
            // the ticket was read before: rows of this block written on other
            // XCDs become visible once this wavefront's caches are invalidated
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
            entered = tw;
        }
        const int64_t b0 = lo + (int64_t)idx * kUnit;
        const int64_t span = (int64_t)take * kUnit;
        const int64_t cnt = hi - b0 < span ? hi - b0 : span;
        const uint32_t ran = take; // units this claim covers
        DebugSink blk = dbg;
        blk.trace = nullptr;
        if (blk.orig)
            blk.orig += b0;
        if constexpr (HALF && KP == 32)
            run_worker_half<KP, T, D, DBG>(Sp + b0, cnt, 2, 0, f, P, Q, lr, lp, lq, blk);
        else if constexpr (HALF)
            run_worker_half<KP, T, D, DBG, false, SKIP>(Sp + b0, cnt, 2, 0, f, P, Q, lr, lp, lq, blk,
                                                        CacheSync{0, false, false}, my_sink);
        else
            run_worker<KP, T, D, DBG, SKIP, false, kCohOff, ATOM>(Sp + b0, cnt, 1, 0, f, P, Q, lr, lp, lq, blk,
                                                                 CacheSync{0, false, false}, my_sink, coh);
        // this wavefront's stores have reached the XCD's L2 before it counts
        // the batches as finished
        __builtin_amdgcn_s_waitcnt(0);
        uint32_t done = 0;
        if (lane == 0)
            done = __hip_atomic_fetch_add(fin + tw, ran, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        done = __builtin_amdgcn_readfirstlane(done);
        if (done + ran == nu) {
            // last batch of the block: every batch's stores are in this XCD's
            // L2; write it back, wait for the write-back, then pass the
            // column on
            release_agent();
            if (lane == 0) {
                if (trace) {
                    stamps[2 * tw + 1] =
                        __hip_atomic_fetch_add(events, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    clocks[2 * tw + 1] = (uint32_t)__builtin_amdgcn_s_memrealtime();
                    __builtin_amdgcn_s_waitcnt(0);
                }
                __hip_atomic_store(tickets + col, (uint32_t)(w + 1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        }
    }
}

// LIBMF's global scheduling table (section 3.2.1), the baseline that
// batch-Hogwild! and wavefront-update replace.  R is cut into an s x s grid;
// every wavefront is one worker; a free worker takes the table's lock, picks
// a block not yet taken this epoch whose row block and column block are both
// unused, marks them used, releases the lock and updates the block's samples
// serially; then it clears its two marks.  An epoch takes every non-empty
// block once.
//
// The blocks not yet taken form a list.  Decision d draws a list position
// from output d of this epoch's stream (high 32 bits times the list length,
// shifted down 32); the holder of the lock checks 64 consecutive list entries
// (cyclically from that position) per step, one per lane, takes the first
// whose row and column are unused and moves the list's last entry into its
// slot.  A single worker therefore takes the blocks in the draw order alone.
//
// Every table word is read and written with agent-scope atomics, which all
// XCDs see coherently; the writes made under the lock have completed
// (s_waitcnt) before the lock is released.  The block's rows are handed over
// between XCDs as in the block-scheduled kernel: the worker writes its L2
// back (agent-scope release) before it clears its marks, and a worker that
// has taken a block invalidates its caches (agent-scope acquire) before it
// reads the rows.
//
// The lock is a ticket lock: a worker draws a ticket once and then only reads
// the serving counter until its turn; the holder passes the lock on to the
// next ticket.  No wavefront leaves while it holds the lock or a block; a
// worker that waits for its turn, or finds no block free, polls (with a
// sleep), and after spin_limit polls in a row raises *err, upon which every
// worker leaves at its next visit to the table (a worker whose ticket is
// never served because its predecessor gave up leaves the same way).
template <int KP, typename T, int D, bool DBG>
__global__ __launch_bounds__(64) void k_table(const Sample* __restrict__ Sp, const int64_t* __restrict__ bstart,
                                              int s, uint32_t nb, uint64_t draw, T* __restrict__ P,
                                              T* __restrict__ Q, float lr, float lp, float lq, int f, uint32_t* tab,
                                              uint32_t spin_limit, int* err, DebugSink dbg, int32_t* trace)
{
    const int lane = lane_id();
    uint32_t* const serving = tab;     // ticket now holding the table
    uint32_t* const left = tab + 1;
    uint32_t* const events = tab + 2;
    uint32_t* const next_ticket = tab + 3;
    uint32_t* const row_used = tab + kTableHdr;
    uint32_t* const col_used = row_used + s;
    uint32_t* const list = col_used + s;
    const uint32_t us = (uint32_t)s;
    uint32_t polls = 0;
    uint32_t ticket = 0;
    bool queued = false;
    for (;;) {
        // take the lock: a ticket lock (first come, first served), so waiting
        // workers only read the serving counter instead of competing in
        // atomic exchanges
        int got = 0, stop = 0;
        if (lane == 0) {
            stop = __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0;
            if (!stop) {
                if (!queued)
                    ticket = __hip_atomic_fetch_add(next_ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                got = __hip_atomic_load(serving, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == ticket;
            }
        }
        if (__builtin_amdgcn_readfirstlane(stop))
            return;
        ticket = __builtin_amdgcn_readfirstlane(ticket);
        queued = true;
        bool wait = !__builtin_amdgcn_readfirstlane(got);
        uint32_t fpos = 0, fblk = 0, d = 0;
        if (!wait) {
            uint32_t rem = 0;
            if (lane == 0)
                rem = __hip_atomic_load(left, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            rem = __builtin_amdgcn_readfirstlane(rem);
            if (rem == 0u) {
                if (lane == 0)
                    __hip_atomic_store(serving, ticket + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                return; // every block has been taken
            }
            d = nb - rem;
            const uint64_t x = sm64_at(draw, (uint64_t)d);
            const uint32_t pos0 = (uint32_t)(((x >> 32) * (uint64_t)rem) >> 32);
            bool found = false;
            for (uint32_t j0 = 0; j0 < rem && !found; j0 += 64) {
                const uint32_t j = j0 + (uint32_t)lane;
                bool ok = false;
                uint32_t pos = 0, blk = 0;
                if (j < rem) {
                    pos = pos0 + j;
                    pos = pos >= rem ? pos - rem : pos;
                    blk = __hip_atomic_load(list + pos, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    ok = __hip_atomic_load(row_used + blk / us, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u &&
                         __hip_atomic_load(col_used + blk % us, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u;
                }
                const uint64_t hit = __builtin_amdgcn_ballot_w64(ok);
                if (hit) {
                    const int l = (int)__builtin_ctzll(hit);
                    fpos = __builtin_amdgcn_readlane(pos, l);
                    fblk = __builtin_amdgcn_readlane(blk, l);
                    found = true;
                }
            }
            if (lane == 0) {
                if (found) {
                    const uint32_t last = __hip_atomic_load(list + rem - 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(list + fpos, last, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(left, rem - 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(row_used + fblk / us, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    __hip_atomic_store(col_used + fblk % us, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    if (DBG && trace) {
                        const uint32_t stamp =
                            __hip_atomic_fetch_add(events, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        trace[3 * (int64_t)d] = (int32_t)fblk;
                        trace[3 * (int64_t)d + 1] = (int32_t)stamp;
                    }
                }
                // every table write has completed before the lock passes on
                __builtin_amdgcn_s_waitcnt(0);
                __hip_atomic_store(serving, ticket + 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            queued = false; // the next attempt takes a new ticket
            wait = !found;
        }
        if (wait) {
            int give_up = 0;
            if (lane == 0 && ++polls > spin_limit) {
                __hip_atomic_fetch_or(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                give_up = 1;
            }
            if (__builtin_amdgcn_readfirstlane(give_up))
                return;
            __builtin_amdgcn_s_sleep(8);
            continue;
        }
        polls = 0;
        // rows of this block written on other XCDs become visible once this
        // wavefront's caches are invalidated
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
        const int64_t lo = bstart[fblk], hi = bstart[fblk + 1];
        DebugSink blk = dbg;
        blk.trace = nullptr;
        if (blk.orig)
            blk.orig += lo;
        run_worker<KP, T, D, DBG, false>(Sp + lo, hi - lo, 1, 0, f, P, Q, lr, lp, lq, blk);
        // the block's stores reach memory before its row and column are free
        __builtin_amdgcn_s_waitcnt(0);
        release_agent();
        if (lane == 0) {
            if (DBG && trace) {
                trace[3 * (int64_t)d + 2] =
                    (int32_t)__hip_atomic_fetch_add(events, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __builtin_amdgcn_s_waitcnt(0);
            }
            __hip_atomic_store(row_used + fblk / us, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            __hip_atomic_store(col_used + fblk % us, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
    }
}

// One wave of the deterministic wavefront-update schedule per launch: the
// cross-check of the ticketed kernel above.  Workgroup i (one wavefront) is
// worker i and updates block (i, sigma_i(w)) serially in array order; the
// blocks of one wave share no row and no column, and the launch boundary
// orders consecutive waves (every write of wave w is visible to wave w + 1
// on any XCD), so no ticket is needed.  Same update code, same per-block
// order, hence the same factors bit for bit.
template <int KP, typename T, int D, bool DBG>
__global__ __launch_bounds__(64) void k_wave(const Sample* __restrict__ Sp, const int64_t* __restrict__ bstart,
                                             int s, int w, uint64_t sigma_c, uint64_t sigma_o, T* __restrict__ P,
                                             T* __restrict__ Q, float lr, float lp, float lq, int f, DebugSink dbg,
                                             int32_t* trace)
{
    __shared__ int Cperm[kMaxGrid], Ooff[kMaxGrid];
    if (threadIdx.x == 0) {
        shuffle_perm(sigma_c, s, Cperm);
        shuffle_perm(sigma_o, s, Ooff);
    }
    __syncthreads();
    const int i = (int)blockIdx.x;
    const int col = Cperm[(i + Ooff[w]) % s];
    const int64_t b = (int64_t)i * s + col;
    const int64_t lo = bstart[b], hi = bstart[b + 1];
    if (trace && threadIdx.x == 0)
        trace[(int64_t)i * s + w] = col;
    DebugSink blk = dbg;
    blk.trace = nullptr;
    if (blk.orig)
        blk.orig += lo;
    run_worker<KP, T, D, DBG, false>(Sp + lo, hi - lo, 1, 0, f, P, Q, lr, lp, lq, blk);
}

template <int KP, typename T, int D>
static int occupancy_blocked_t(int threads, bool half)
{
    int blocks = 0;
    if constexpr (KP == 32) {
        if (half) // the only variant such launches use
            return hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_blocked<KP, T, D, false, false, true>,
                                                                threads, 0) == hipSuccess
                       ? blocks
                       : 0;
    } else if constexpr (kHalfRows<KP, T>) {
        if (half) { // both variants such launches may use
            int skip = 0;
            if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_blocked<KP, T, D, false, false, true>, threads,
                                                             0) != hipSuccess ||
                hipOccupancyMaxActiveBlocksPerMultiprocessor(&skip, k_blocked<KP, T, D, false, true, true>, threads,
                                                             0) != hipSuccess)
                return 0;
            return blocks < skip ? blocks : skip;
        }
    }
    // the co-residency cap must hold for both variants the launcher may pick
    int plain = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_blocked<KP, T, D, false, true>, threads, 0) !=
            hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&plain, k_blocked<KP, T, D, false, false>, threads, 0) !=
            hipSuccess)
        return 0;
    return blocks < plain ? blocks : plain;
}

template <int KP, typename T>
static int occupancy_blocked_kp(int depth, int threads, bool half)
{
    switch (depth) {
    case 1: return occupancy_blocked_t<KP, T, 1>(threads, half);
    case 2: return occupancy_blocked_t<KP, T, 2>(threads, half);
    case 4: return occupancy_blocked_t<KP, T, 4>(threads, half);
    case 8: return occupancy_blocked_t<KP, T, 8>(threads, half);
    default: return 0;
    }
}

// Test RMSE, pass 1 (section 3.2.4): wavefront w of kRmseWaves sums the
// squared errors of its contiguous share of the test samples in binary64.
// Samples are independent here, so 8 are fetched before any is reduced.
template <int KP, typename T>
__global__ __launch_bounds__(256) void k_rmse_partial(const Sample* __restrict__ S, int64_t ntest,
                                                      const T* __restrict__ P, const T* __restrict__ Q,
                                                      double* __restrict__ partial)
{
    constexpr int E = Geo<KP>::E;
    constexpr int A = Geo<KP>::A;
    constexpr int U = 8;
    typedef Row<T, E> R;
    const int lane = lane_id();
    const bool holds = (A == 64) || (lane < A);
    const int col = lane * E;
    const int64_t wave = uniform64((int64_t)blockIdx.x * 4 + (threadIdx.x >> 6));
    const int64_t share = (ntest + kRmseWaves - 1) / kRmseWaves;
    const int64_t lo = wave * share;
    const int64_t hi = lo + share < ntest ? lo + share : ntest;
    double acc = 0.0;
    for (int64_t c0 = lo; c0 < hi; c0 += 64) {
        const int cnt = (int)(hi - c0 >= 64 ? 64 : hi - c0);
        int cu = 0, cv = 0;
        float cr = 0.f;
        if (lane < cnt) {
            cu = __builtin_nontemporal_load(&S[c0 + lane].u);
            cv = __builtin_nontemporal_load(&S[c0 + lane].v);
            cr = __builtin_nontemporal_load(&S[c0 + lane].r);
        }
        for (int i0 = 0; i0 < cnt; i0 += U) {
            float p[U][E], q[U][E];
#pragma unroll
            for (int j = 0; j < U; ++j) {
                const int i = i0 + j;
#pragma unroll
                for (int e = 0; e < E; ++e)
                    p[j][e] = q[j][e] = 0.f;
                if (i < cnt && holds) {
                    const int u = __builtin_amdgcn_readlane(cu, i);
                    const int v = __builtin_amdgcn_readlane(cv, i);
                    R::load(P + (int64_t)u * KP + col, p[j]);
                    R::load(Q + (int64_t)v * KP + col, q[j]);
                }
            }
#pragma unroll
            for (int j = 0; j < U; ++j) {
                const int i = i0 + j;
                float dot = 0.f;
#pragma unroll
                for (int e = 0; e < E; ++e)
                    dot += p[j][e] * q[j][e];
                dot = wave_sum(dot);
                if (i < cnt) {
                    const float r = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cr), i));
                    const double e = (double)(r - dot);
                    acc += e * e;
                }
            }
        }
    }
    if (lane == 0)
        partial[wave] = acc;
}

template <int KP, typename T, int D, bool DBG>
static hipError_t launch_epoch_d(const EpochLaunch& a, hipStream_t st)
{
    T* P = (T*)a.P;
    T* Q = (T*)a.Q;
    if (a.scheme == kSchemeHogwild) {
        const DebugSink dbg{a.visits, nullptr, a.trace_batch};
        if constexpr (kHalfRows<KP, T>) {
            if (a.half) {
                const int64_t blocks = ((a.W + 1) / 2 + 3) / 4;
                if constexpr (sizeof(T) * KP == 4 * 32 && !DBG) { // one dword of a row per lane
                    if (a.buf) {
                        hipLaunchKernelGGL((k_hogwild_half<KP, T, D, false, true>), dim3((unsigned)blocks),
                                           dim3(kHogwildBlock), 0, st, a.S, a.nnz, a.W, a.f, P, Q, a.lr, a.lp, a.lq,
                                           dbg, a.sync_every, a.sync_l1, a.nx);
                        return hipGetLastError();
                    }
                }
                hipLaunchKernelGGL((k_hogwild_half<KP, T, D, DBG>), dim3((unsigned)blocks), dim3(kHogwildBlock), 0,
                                   st, a.S, a.nnz, a.W, a.f, P, Q, a.lr, a.lp, a.lq, dbg, a.sync_every, a.sync_l1,
                                   a.nx);
                return hipGetLastError();
            }
        }
        const int64_t blocks = (a.W + 3) / 4;
        const Coherence coh{a.hot_p, a.hot_q, a.coh_p != 0, a.coh_q != 0};
        if constexpr (D == 1 && (sizeof(T) == 4 || Geo<KP>::E % 2 == 0)) {
            if (a.atomic) {
                // atomic row updates over the whole GPU; with coh == kCohBoth the
                // rows are also read with agent-scope loads
                if (a.coh == kCohBoth)
                    hipLaunchKernelGGL((k_hogwild<KP, T, 1, DBG, false, kCohBoth, true>), dim3((unsigned)blocks),
                                       dim3(kHogwildBlock), 0, st, a.S, a.nnz, a.W, a.f, P, Q, a.lr, a.lp, a.lq, dbg,
                                       a.sync_every, a.sync_l1, a.nx, coh);
                else
                    hipLaunchKernelGGL((k_hogwild<KP, T, 1, DBG, false, kCohOff, true>), dim3((unsigned)blocks),
                                       dim3(kHogwildBlock), 0, st, a.S, a.nnz, a.W, a.f, P, Q, a.lr, a.lp, a.lq, dbg,
                                       a.sync_every, a.sync_l1, a.nx, coh);
                return hipGetLastError();
            }
        }
        if (a.atomic)
            return hipErrorInvalidValue;
        if (a.coh != kCohOff) {
#define MFSGD_COH_LAUNCH(C)                                                                                        \
    hipLaunchKernelGGL((k_hogwild<KP, T, D, DBG, false, C>), dim3((unsigned)blocks), dim3(kHogwildBlock), 0, st,   \
                       a.S, a.nnz, a.W, a.f, P, Q, a.lr, a.lp, a.lq, dbg, a.sync_every, a.sync_l1, a.nx, coh)
            switch (a.coh) {
            case kCohStore: MFSGD_COH_LAUNCH(kCohStore); break;
            case kCohBoth: MFSGD_COH_LAUNCH(kCohBoth); break;
            case kCohNT: MFSGD_COH_LAUNCH(kCohNT); break;
            case kCohSys: MFSGD_COH_LAUNCH(kCohSys); break;
            default: return hipErrorInvalidValue;
            }
#undef MFSGD_COH_LAUNCH
            return hipGetLastError();
        }
        constexpr bool kDword = sizeof(T) * Geo<KP>::E == 4; // one dword of a row per lane
        if constexpr (kDword && !DBG) {
            if (a.buf) {
                hipLaunchKernelGGL((k_hogwild<KP, T, D, false, true>), dim3((unsigned)blocks), dim3(kHogwildBlock), 0,
                                   st, a.S, a.nnz, a.W, a.f, P, Q, a.lr, a.lp, a.lq, dbg, a.sync_every, a.sync_l1,
                                   a.nx, coh);
                return hipGetLastError();
            }
        }
        hipLaunchKernelGGL((k_hogwild<KP, T, D, DBG>), dim3((unsigned)blocks), dim3(kHogwildBlock), 0, st, a.S,
                           a.nnz, a.W, a.f, P, Q, a.lr, a.lp, a.lq, dbg, a.sync_every, a.sync_l1, a.nx, coh);
    } else if (a.scheme == kSchemeWaveLaunch) {
        const DebugSink dbg{a.visits, a.orig, nullptr};
        hipLaunchKernelGGL((k_wave<KP, T, D, DBG>), dim3((unsigned)a.s), dim3(64), 0, st, a.S, a.bstart, a.s, a.wave,
                           a.sigma_c, a.sigma_o, P, Q, a.lr, a.lp, a.lq, a.f, dbg, a.trace_wave);
    } else {
        const DebugSink dbg{a.visits, a.orig, nullptr};
        const Coherence acoh{a.hot_p, a.hot_q, false, false};
        if constexpr (KP == 32) {
            if (a.half && !a.sink) {
                hipLaunchKernelGGL((k_blocked<KP, T, D, DBG, false, true>), dim3((unsigned)a.grid),
                                   dim3(64 * a.wg_waves), 0, st, a.S, a.bstart, a.s, a.xslots, a.tmap, a.xteams, a.nx, a.pool, a.prio,
                                   a.free_run, a.sigma_c, a.sigma_o, a.tail, P, Q, a.lr, a.lp, a.lq, a.f, a.tickets, a.sched,
                                   a.spin_limit, a.err, dbg, a.trace_wave, (T*)nullptr, acoh);
                return hipGetLastError();
            }
        }
        if constexpr (KP > 32 && kHalfRows<KP, T>) {
            if (a.half) {
                // two batches per claim at wider rows (option half_waves = 2),
                // with skipped stores where the plan calls for them (never in
                // epochs with debug output)
                if (!DBG && a.sink)
                    hipLaunchKernelGGL((k_blocked<KP, T, D, false, true, true>), dim3((unsigned)a.grid),
                                       dim3(64 * a.wg_waves), 0, st, a.S, a.bstart, a.s, a.xslots, a.tmap, a.xteams, a.nx,
                                       a.pool, a.prio, a.free_run, a.sigma_c, a.sigma_o, a.tail, P, Q, a.lr, a.lp, a.lq, a.f,
                                       a.tickets, a.sched, a.spin_limit, a.err, dbg, a.trace_wave, (T*)a.sink, acoh);
                else
                    hipLaunchKernelGGL((k_blocked<KP, T, D, DBG, false, true>), dim3((unsigned)a.grid),
                                       dim3(64 * a.wg_waves), 0, st, a.S, a.bstart, a.s, a.xslots, a.tmap, a.xteams, a.nx,
                                       a.pool, a.prio, a.free_run, a.sigma_c, a.sigma_o, a.tail, P, Q, a.lr, a.lp, a.lq, a.f,
                                       a.tickets, a.sched, a.spin_limit, a.err, dbg, a.trace_wave, (T*)nullptr, acoh);
                return hipGetLastError();
            }
        }
        if constexpr (D == 1 && (sizeof(T) == 4 || Geo<KP>::E % 2 == 0)) {
            if (a.atomic) {
                hipLaunchKernelGGL((k_blocked<KP, T, 1, DBG, false, false, true>), dim3((unsigned)a.grid),
                                   dim3(64 * a.wg_waves), 0, st, a.S, a.bstart, a.s, a.xslots, a.tmap, a.xteams, a.nx, a.pool, a.prio,
                                   a.free_run, a.sigma_c, a.sigma_o, a.tail, P, Q, a.lr, a.lp, a.lq, a.f, a.tickets, a.sched,
                                   a.spin_limit, a.err, dbg, a.trace_wave, (T*)nullptr, acoh);
                return hipGetLastError();
            }
        }
        if (a.atomic)
            return hipErrorInvalidValue;
        // skipped stores only in epochs without debug output (they never change results)
        if (!DBG && a.sink)
            hipLaunchKernelGGL((k_blocked<KP, T, D, false, true>), dim3((unsigned)a.grid), dim3(64 * a.wg_waves), 0,
                               st, a.S, a.bstart, a.s, a.xslots, a.tmap, a.xteams, a.nx, a.pool, a.prio, a.free_run, a.sigma_c, a.sigma_o, a.tail, P, Q,
                               a.lr, a.lp, a.lq, a.f, a.tickets, a.sched, a.spin_limit, a.err, dbg, a.trace_wave,
                               (T*)a.sink, acoh);
        else
            hipLaunchKernelGGL((k_blocked<KP, T, D, DBG, false>), dim3((unsigned)a.grid), dim3(64 * a.wg_waves), 0,
                               st, a.S, a.bstart, a.s, a.xslots, a.tmap, a.xteams, a.nx, a.pool, a.prio, a.free_run, a.sigma_c, a.sigma_o, a.tail, P, Q,
                               a.lr, a.lp, a.lq, a.f, a.tickets, a.sched, a.spin_limit, a.err, dbg, a.trace_wave,
                               (T*)nullptr, acoh);
    }
    return hipGetLastError();
}

template <int KP, typename T, int D>
static hipError_t launch_epoch_t(const EpochLaunch& a, hipStream_t st)
{
    if (a.visits || a.trace_batch)
        return launch_epoch_d<KP, T, D, true>(a, st);
    return launch_epoch_d<KP, T, D, false>(a, st);
}

template <int KP, typename T>
static hipError_t launch_epoch_kp(const EpochLaunch& a, hipStream_t st)
{
    switch (a.depth) {
    case 1: return launch_epoch_t<KP, T, 1>(a, st);
    case 2: return launch_epoch_t<KP, T, 2>(a, st);
    case 4: return launch_epoch_t<KP, T, 4>(a, st);
    case 8: return launch_epoch_t<KP, T, 8>(a, st);
    default: return hipErrorInvalidValue;
    }
}

template <int KP, typename T, int D>
static hipError_t launch_table_t(const TableLaunch& a, hipStream_t st)
{
    if (a.nb == 0)
        return hipSuccess;
    const dim3 grid((unsigned)a.W), block(64);
    if (a.visits || a.trace) {
        const DebugSink dbg{a.visits, a.orig, nullptr};
        hipLaunchKernelGGL((k_table<KP, T, D, true>), grid, block, 0, st, a.Sp, a.bstart, a.s, a.nb, a.draw, (T*)a.P,
                           (T*)a.Q, a.lr, a.lp, a.lq, a.f, a.tab, a.spin_limit, a.err, dbg, a.trace);
    } else {
        const DebugSink dbg{nullptr, nullptr, nullptr};
        hipLaunchKernelGGL((k_table<KP, T, D, false>), grid, block, 0, st, a.Sp, a.bstart, a.s, a.nb, a.draw,
                           (T*)a.P, (T*)a.Q, a.lr, a.lp, a.lq, a.f, a.tab, a.spin_limit, a.err, dbg,
                           (int32_t*)nullptr);
    }
    return hipGetLastError();
}

template <int KP, typename T>
static hipError_t launch_table_kp(const TableLaunch& a, hipStream_t st)
{
    switch (a.depth) {
    case 1: return launch_table_t<KP, T, 1>(a, st);
    case 2: return launch_table_t<KP, T, 2>(a, st);
    case 4: return launch_table_t<KP, T, 4>(a, st);
    case 8: return launch_table_t<KP, T, 8>(a, st);
    default: return hipErrorInvalidValue;
    }
}

// wavefronts of the one-address-space batch-Hogwild! kernel resident per CU
template <int KP, typename T, int D>
static int occupancy_t(bool half)
{
    int blocks = 0;
    hipError_t e;
    if constexpr (kHalfRows<KP, T>) {
        if (half)
            e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_hogwild_half<KP, T, D, false>, kHogwildBlock,
                                                             0);
        else
            e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_hogwild<KP, T, D, false>, kHogwildBlock, 0);
    } else {
        e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_hogwild<KP, T, D, false>, kHogwildBlock, 0);
    }
    if (e != hipSuccess)
        return 0;
    return blocks * (kHogwildBlock / 64);
}

template <int KP, typename T>
static int occupancy_kp(int depth, bool half)
{
    switch (depth) {
    case 1: return occupancy_t<KP, T, 1>(half);
    case 2: return occupancy_t<KP, T, 2>(half);
    case 4: return occupancy_t<KP, T, 4>(half);
    case 8: return occupancy_t<KP, T, 8>(half);
    default: return 0;
    }
}

template <typename T>
__global__ void k_init(T* __restrict__ A, int64_t rows, int k, int KP, uint64_t stream, double inv_sqrt_k)
{
    const int64_t total = rows * KP;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t row = i / KP;
        const int j = (int)(i - row * KP);
        double val = 0.0;
        if (j < k) {
            const uint64_t x = sm64_at(stream, (uint64_t)(row * k + j));
            val = (double)(x >> 40) * 0x1p-24 * inv_sqrt_k;
        }
        A[i] = from_f64<T>(val);
    }
}

template <typename T>
struct Dispatch {
    static hipError_t epoch(const EpochLaunch& a, hipStream_t st)
    {
        switch (a.KP) {
        case 32: return launch_epoch_kp<32, T>(a, st);
        case 64: return launch_epoch_kp<64, T>(a, st);
        case 128: return launch_epoch_kp<128, T>(a, st);
        case 256: return launch_epoch_kp<256, T>(a, st);
        case 512: return launch_epoch_kp<512, T>(a, st);
        default: return hipErrorInvalidValue;
        }
    }
    static hipError_t table_epoch(const TableLaunch& a, hipStream_t st)
    {
        switch (a.KP) {
        case 32: return launch_table_kp<32, T>(a, st);
        case 64: return launch_table_kp<64, T>(a, st);
        case 128: return launch_table_kp<128, T>(a, st);
        case 256: return launch_table_kp<256, T>(a, st);
        case 512: return launch_table_kp<512, T>(a, st);
        default: return hipErrorInvalidValue;
        }
    }
    static int occupancy(int KP, int depth, bool half)
    {
        switch (KP) {
        // half: the two-workers-per-wavefront kernel wherever it runs (its
        // lanes hold twice the values, so fewer of its wavefronts fit a CU)
        case 32: return occupancy_kp<32, T>(depth, half);
        case 64: return occupancy_kp<64, T>(depth, half);
        case 128: return occupancy_kp<128, T>(depth, half);
        case 256: return occupancy_kp<256, T>(depth, half);
        case 512: return occupancy_kp<512, T>(depth, half);
        default: return 0;
        }
    }
    static int occupancy_blocked(int KP, int depth, int threads, bool half)
    {
        // half: two batches per claim, at every width whose half-wavefront
        // rows fit (the variant holds twice the values per lane)
        switch (KP) {
        case 32: return occupancy_blocked_kp<32, T>(depth, threads, half);
        case 64: return occupancy_blocked_kp<64, T>(depth, threads, half);
        case 128: return occupancy_blocked_kp<128, T>(depth, threads, half);
        case 256: return occupancy_blocked_kp<256, T>(depth, threads, half);
        case 512: return occupancy_blocked_kp<512, T>(depth, threads, half);
        default: return 0;
        }
    }
    static hipError_t rmse(int KP, const Sample* S, int64_t ntest, const void* P, const void* Q, double* partial,
                           hipStream_t st)
    {
        const dim3 grid(kRmseWaves / 4), block(256);
        switch (KP) {
        case 32: hipLaunchKernelGGL((k_rmse_partial<32, T>), grid, block, 0, st, S, ntest, (const T*)P, (const T*)Q, partial); break;
        case 64: hipLaunchKernelGGL((k_rmse_partial<64, T>), grid, block, 0, st, S, ntest, (const T*)P, (const T*)Q, partial); break;
        case 128: hipLaunchKernelGGL((k_rmse_partial<128, T>), grid, block, 0, st, S, ntest, (const T*)P, (const T*)Q, partial); break;
        case 256: hipLaunchKernelGGL((k_rmse_partial<256, T>), grid, block, 0, st, S, ntest, (const T*)P, (const T*)Q, partial); break;
        case 512: hipLaunchKernelGGL((k_rmse_partial<512, T>), grid, block, 0, st, S, ntest, (const T*)P, (const T*)Q, partial); break;
        default: return hipErrorInvalidValue;
        }
        return hipGetLastError();
    }
    static hipError_t init(void* A, int64_t rows, int k, int KP, uint64_t stream, double inv_sqrt_k, hipStream_t st)
    {
        const int64_t total = rows * KP;
        int64_t blocks = (total + 255) / 256;
        if (blocks > 65536)
            blocks = 65536;
        hipLaunchKernelGGL((k_init<T>), dim3((unsigned)blocks), dim3(256), 0, st, (T*)A, rows, k, KP, stream,
                           inv_sqrt_k);
        return hipGetLastError();
    }
};

} // namespace mfsgd
