// One eviction step of the DeltaS retention policy (Section 3.3, Algorithm 1).
//
// kv_select (one workgroup of 1024 threads) turns the cache metadata into a
// keep list without any host round trip:
//   * sinks = first n_sink slots, window = last n_window slots, the rest are
//     candidates;
//   * the candidates form runs of equal chunk id (the cache is in arrival
//     order), each run shares one score; a run's key is
//     (orderable(score), chunk id), bigger = better, unique per run;
//   * span of a run: floor(N (a - a_min) / (a_max - a_min + 1)); each span
//     keeps min(len, quota - (tokens of better runs in the span)) of every run,
//     newest tokens first (ties within a chunk go to the newer position);
//   * the leftover budget is filled the same way over all spans from the
//     tokens not yet kept;
//   * kept slots -> ascending keep list and its inverse on [0, M).
// Slot data is read in blocks of 4 consecutive slots per thread with one
// 16-byte load (adjacent lanes read adjacent 16 bytes), 4 Ki slots per
// block and memory round trip.
// With a slot table (the indexed variant) the K and V rows never move: the
// select kernel itself compacts pos, chunk_id and slot (the physical row of
// each logical token) in place and lists the freed physical rows.
// The kept rows then move down in place: slot d receives row keep[d]
// (keep[d] >= d); the shift keep[d] - d never decreases with d.
// kv_gather handles the destinations whose shift is large.  Writing slot d is
// safe once the reader of row d -- the destination inv[d] < d, if row d is
// kept -- has its data in registers.  Workgroups take increasing tickets,
// signal "read done" before they wait, and only ever wait on lower tickets,
// so every wait ends; the wait is also bounded and reports a timeout in the
// status word instead of hanging.  Its parallelism is the shift itself (only
// rows a shift apart are independent), so destinations with a small shift
// (fewer than STAGE_BYTES of rows) go first through kv_stage instead: blocks
// of destinations are copied to a staging area and back in two launches,
// with no waits at all (a block only reads at or above its own start, and
// the blocks run in order).
#include <algorithm>
#include <mutex>

#include "common.h"
#include "kernels.h"

namespace ds {

constexpr int SEL_THREADS = 1024;
constexpr int SEL_PER = 4;                          // consecutive slots per thread per pass block
constexpr int SEL_BLOCK = SEL_THREADS * SEL_PER;
static_assert(SEL_PER == 4, "pass 2 stores a thread's four inverse entries as one int4");
constexpr int GATHER_U = 16;                        // uint4 per thread per group
constexpr int SPIN_LIMIT = 1 << 22;
constexpr long long STAGE_BYTES = 64ll << 20;       // below this much shift, rows are staged
constexpr long long STAGE_AREA = 256ll << 20;       // staging area of one block of destinations
constexpr int STAGE_WG = 1024;                      // workgroups per staging launch (each loops over rows)

// pointer into global memory (lets the compiler emit global rather than flat accesses)
#define GPTR(T) __attribute__((address_space(1))) T *
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct KvArgs {
    int32_t *pos;    // written only by the indexed variant
    int32_t *chunk;
    const float *scores;
    int num_chunks, len, M, n_s, n_w, N;
    int n_flags, n_chunks;
    int stage_shift;   // destinations with keep[d] - d below this are staged
    int32_t *status;   // [0] outcome (0 ok, 1 invariants broken, 2 keep count wrong, 3 gather wait timed
                       // out), [1] skip or stop the moves, [2] wait timed out, [3] first moved slot,
                       // [4] first slot moved by the ticket gather (the staged ones lie in [3], [4])
    uint32_t *ticket;
    int32_t *keep, *inv, *run_start, *run_bkt, *run_take, *run_from, *th_run;
    unsigned long long *run_key;
    int32_t *flags;
    int32_t *keep_out;
    int32_t *slot;      // indexed variant: physical row of each logical token (NULL: gather variant)
    int32_t *free_out;  // indexed variant: physical rows of the evicted tokens
    int32_t *outcome_out;  // indexed variant: a copy of status[0] for the caller (or NULL)
    char **plane_tab;  // device copy of the plane pointers, read by the gather
    char *planes[KV_MAX_PLANES];
    int n_planes;
};

__device__ __forceinline__ uint32_t orderable(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Barrier that orders LDS only: the block reductions below exchange partial
// sums through LDS, and a full __syncthreads would also wait for every global
// store in flight (the keep list written in the same loop).
__device__ __forceinline__ void lds_sync() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Exclusive prefix sum over the 1024 threads of the block.
// Inclusive prefix sum over the 64 lanes of a wave with DPP moves: row
// shifts by 1, 2, 4, 8 within each row of 16 lanes, then the last lane of a
// row added to the next row(s) by row broadcasts (rows 1 and 3 get lane 15,
// rows 2 and 3 lane 31).  Lanes without a source add 0.
__device__ __forceinline__ int wave_incl_scan(int v) {
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);  // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);  // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);  // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);  // row_shr:8
    v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);  // row_bcast:15 into rows 1, 3
    v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);  // row_bcast:31 into rows 2, 3
    return v;
}

// Exclusive prefix sum over the 1024 threads of the block: a scan inside each
// wave, then wave 0 scans the 16 wave totals the same way.
__device__ int block_excl_scan(int x, int *s_tmp, int &total) {
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int incl = wave_incl_scan(x);
    if (lane == 63) s_tmp[wid] = incl;
    lds_sync();
    if (wid == 0) {
        const int t = lane < SEL_THREADS / 64 ? s_tmp[lane] : 0;
        const int it = wave_incl_scan(t);
        if (lane < SEL_THREADS / 64) s_tmp[lane] = it - t;
        if (lane == SEL_THREADS / 64 - 1) s_tmp[SEL_THREADS / 64] = it;
    }
    lds_sync();
    const int res = s_tmp[wid] + incl - x;
    total = s_tmp[SEL_THREADS / 64];
    lds_sync();
    return res;
}

// Same DPP pattern with max; lanes without a source contribute -1 (x >= -1).
__device__ __forceinline__ int wave_incl_max(int v) {
    v = max(v, __builtin_amdgcn_update_dpp(-1, v, 0x111, 0xf, 0xf, false));
    v = max(v, __builtin_amdgcn_update_dpp(-1, v, 0x112, 0xf, 0xf, false));
    v = max(v, __builtin_amdgcn_update_dpp(-1, v, 0x114, 0xf, 0xf, false));
    v = max(v, __builtin_amdgcn_update_dpp(-1, v, 0x118, 0xf, 0xf, false));
    v = max(v, __builtin_amdgcn_update_dpp(-1, v, 0x142, 0xa, 0xf, false));
    v = max(v, __builtin_amdgcn_update_dpp(-1, v, 0x143, 0xc, 0xf, false));
    return v;
}

// Maximum of x over the lower threads of the block (-1 for thread 0); x >= -1.
__device__ int block_excl_max(int x, int *s_tmp) {
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    const int incl = wave_incl_max(x);
    const int excl = __shfl(incl, max(lane - 1, 0), 64);
    if (lane == 63) s_tmp[wid] = incl;
    lds_sync();
    if (wid == 0) {
        const int t = lane < SEL_THREADS / 64 ? s_tmp[lane] : -1;
        const int it = wave_incl_max(t);
        const int et = __shfl(it, max(lane - 1, 0), 64);
        if (lane < SEL_THREADS / 64) s_tmp[lane] = lane > 0 ? et : -1;
    }
    lds_sync();
    const int res = max(s_tmp[wid], lane > 0 ? excl : -1);
    lds_sync();
    return res;
}

__device__ long long block_sum_ll(long long x, long long *s_tmp) {
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
    if (lane == 0) s_tmp[wid] = x;
    lds_sync();
    if (tid == 0) {
        long long acc = 0;
        for (int i = 0; i < SEL_THREADS / 64; ++i) acc += s_tmp[i];
        s_tmp[SEL_THREADS / 64] = acc;
    }
    lds_sync();
    const long long r = s_tmp[SEL_THREADS / 64];
    lds_sync();
    return r;
}

// SEL_PER consecutive int32 from [lo, lo + SEL_PER); entries at or past len read as 0.
__device__ __forceinline__ void load_block(const int32_t *p, int lo, int len, int (&out)[SEL_PER]) {
    if (lo + SEL_PER <= len) {
#pragma unroll
        for (int q = 0; q < SEL_PER / 4; ++q) {
            const int4 v = *(const int4 *)(p + lo + 4 * q);
            out[4 * q] = v.x;
            out[4 * q + 1] = v.y;
            out[4 * q + 2] = v.z;
            out[4 * q + 3] = v.w;
        }
    } else {
#pragma unroll
        for (int k = 0; k < SEL_PER; ++k) out[k] = (lo + k < len) ? p[lo + k] : 0;
    }
}

struct RunRec {
    unsigned long long key;  // (orderable score, chunk id): bigger is better
    int len;                 // candidate slots of the run
    int bkt;                 // span of the run
};
constexpr int RUN_CAP = 2048;  // runs ranked from LDS
constexpr int SORT_MIN = 512;  // more runs than this (up to RUN_CAP) are ranked by sorting

__global__ __launch_bounds__(SEL_THREADS) void kv_select_kernel(KvArgs a) {
    __shared__ RunRec s_run[RUN_CAP];
    __shared__ int s_take[RUN_CAP], s_from[RUN_CAP], s_ord[RUN_CAP];
    __shared__ int s_keep[SEL_BLOCK], s_free[SEL_BLOCK];  // one pass-2 block's keep entries and freed slots
    __shared__ int s_scan[SEL_THREADS / 64 + 1];
    __shared__ long long s_ll[SEL_THREADS / 64 + 1];
    __shared__ int s_bad;
    const int tid = threadIdx.x;

    if (tid == 0) {
        a.status[0] = 0;
        a.status[1] = 0;
        a.status[2] = 0;
        *a.ticket = 0u;
        s_bad = 0;
    }
    // copy of the plane table with constant indices (no dynamic indexing of
    // the kernel-argument array)
#pragma unroll
    for (int p = 0; p < KV_MAX_PLANES; ++p)
        if (p == tid && p < a.n_planes) a.plane_tab[p] = a.planes[p];

    const int c0 = a.n_s, c1 = a.len - a.n_w;

    // ---- pass 1: cache invariants and runs of equal chunk id among the
    // candidates [c0, c1); th_run[block][thread] = runs starting before the
    // thread's slots
    int R = 0;
    // the next block's entries are loaded while this one is scanned
    int nch[SEL_PER], nps[SEL_PER], npc = -1, npp = 0;
    auto fetch1 = [&](int base) {
        const int lo = base + tid * SEL_PER;
        load_block(a.chunk, lo, a.len, nch);
        load_block(a.pos, lo, a.len, nps);
        const bool has_prev = lo > 0 && lo <= a.len;
        npc = has_prev ? a.chunk[lo - 1] : -1;
        npp = has_prev ? a.pos[lo - 1] : 0;
    };
    if (a.len > 0) fetch1(0);
    for (int base = 0; base < a.len; base += SEL_BLOCK) {
        const int lo = base + tid * SEL_PER;
        int ch[SEL_PER], ps[SEL_PER];
#pragma unroll
        for (int k = 0; k < SEL_PER; ++k) {
            ch[k] = nch[k];
            ps[k] = nps[k];
        }
        const int pc0 = npc;
        int pc = pc0, pp = npp;
        if (base + SEL_BLOCK < a.len) fetch1(base + SEL_BLOCK);
        int bad = 0, cnt = 0;
#pragma unroll
        for (int k = 0; k < SEL_PER; ++k) {
            const int i = lo + k;
            if (i < a.len) {
                if (ch[k] < 0 || ch[k] >= a.num_chunks) bad = 1;
                if (i > 0 && (ch[k] < pc || ps[k] <= pp)) bad = 1;
                if (i >= c0 && i < c1 && (i == c0 || ch[k] != pc)) ++cnt;
                pc = ch[k];
                pp = ps[k];
            }
        }
        if (bad) atomicOr(&s_bad, 1);
        int tot = 0;
        int off = R + block_excl_scan(cnt, s_scan, tot);
        a.th_run[base / SEL_PER + tid] = off;
        pc = pc0;
#pragma unroll
        for (int k = 0; k < SEL_PER; ++k) {
            const int i = lo + k;
            if (i < a.len) {
                if (i >= c0 && i < c1 && (i == c0 || ch[k] != pc)) a.run_start[off++] = i;
                pc = ch[k];
            }
        }
        R += tot;
    }
    __syncthreads();
    if (s_bad) {
        if (tid == 0) {
            a.status[0] = 1;
            a.status[1] = 1;
            if (a.outcome_out) *a.outcome_out = 1;
        }
        return;
    }
    if (tid == 0) a.run_start[R] = c1;
    __syncthreads();

    // ---- run keys and spans.  The two ranking passes below compare every run
    // with every other; up to RUN_CAP runs they read a copy of the run table
    // in LDS (one 16-byte read per comparison), beyond that the global one.
    const int ncand = c1 - c0;
    const int a_min = (ncand > 0) ? a.chunk[c0] : 0;
    const int a_max = (ncand > 0) ? a.chunk[c1 - 1] : 0;
    const long long span = (long long)a_max - a_min + 1;
    const int N = max(1, a.N);
    const bool in_lds = R <= RUN_CAP;
    for (int r = tid; r < R; r += SEL_THREADS) {
        const int rs = a.run_start[r], re = a.run_start[r + 1];
        const int chn = a.chunk[rs];
        const unsigned long long key = ((unsigned long long)orderable(a.scores[chn]) << 32) | (unsigned)chn;
        const int bkt = (int)(((long long)N * (chn - a_min)) / span);
        a.run_key[r] = key;
        a.run_bkt[r] = bkt;
        if (in_lds) s_run[r] = RunRec{key, re - rs, bkt};
    }
    __syncthreads();

    // ---- ranking.  Every run is compared with every other (from the LDS
    // copy up to RUN_CAP runs, else in global memory), except from SORT_MIN to
    // RUN_CAP runs: there the run indices are sorted in LDS (bitonic network;
    // keys are unique, one run per chunk id) and what a run keeps follows from
    // prefix sums over the runs ranked above it.  (Per pass on MI355X: 1024
    // runs compared pairwise take ~230k clocks, sorted ~70k; 17 runs
    // pairwise a few hundred.)
    const bool by_sort = in_lds && R > SORT_MIN;
    int Rp = 1;
    while (Rp < R) Rp <<= 1;
    auto sort_runs = [&](auto before) __attribute__((always_inline)) {
        for (int i = tid; i < Rp; i += SEL_THREADS) s_ord[i] = i;
        lds_sync();
        for (int k = 2; k <= Rp; k <<= 1)
            for (int j = k >> 1; j > 0; j >>= 1) {
                for (int q = tid; q < Rp / 2; q += SEL_THREADS) {
                    const int i = ((q & ~(j - 1)) << 1) | (q & (j - 1)), l = i + j;
                    const int x = s_ord[i], y = s_ord[l];
                    if ((i & k) == 0 ? before(y, x) : before(x, y)) {
                        s_ord[i] = y;
                        s_ord[l] = x;
                    }
                }
                lds_sync();
            }
    };
    // sorted positions 2 tid and 2 tid + 1 (Rp <= 2 SEL_THREADS); -1 past R
    const int i0 = 2 * tid, i1 = i0 + 1;
    int tot = 0;

    // ---- per-span quota: a run keeps what the better runs of its span left
    const long long quota = (a.M - a.n_s - a.n_w) / N;
    long long taken = 0;
    if (by_sort) {
        sort_runs([&](int x, int y) {  // x ranks before y: span ascending, key descending
            if (x >= R) return false;
            if (y >= R) return true;
            const RunRec rx = s_run[x], ry = s_run[y];
            return rx.bkt < ry.bkt || (rx.bkt == ry.bkt && rx.key > ry.key);
        });
        const int r0 = i0 < R ? s_ord[i0] : -1, r1 = i1 < R ? s_ord[i1] : -1;
        const int l0 = r0 >= 0 ? s_run[r0].len : 0, l1 = r1 >= 0 ? s_run[r1].len : 0;
        const int b0 = r0 >= 0 ? s_run[r0].bkt : -1, b1 = r1 >= 0 ? s_run[r1].bkt : -1;
        const int bp = (i0 > 0 && i0 <= R) ? s_run[s_ord[i0 - 1]].bkt : -2;
        // slots of the runs ranked before, and where the run's span starts
        const int e0 = block_excl_scan(l0 + l1, s_scan, tot), e1 = e0 + l0;
        const int h0 = (r0 >= 0 && b0 != bp) ? e0 : -1, h1 = (r1 >= 0 && b1 != b0) ? e1 : -1;
        const int hp0 = max(block_excl_max(max(h0, h1), s_scan), h0), hp1 = max(hp0, h1);
        if (r0 >= 0) {
            const int t = (int)min((long long)l0, max(0LL, quota - (e0 - hp0)));
            s_take[r0] = t;
            a.run_take[r0] = t;
            taken += t;
        }
        if (r1 >= 0) {
            const int t = (int)min((long long)l1, max(0LL, quota - (e1 - hp1)));
            s_take[r1] = t;
            a.run_take[r1] = t;
            taken += t;
        }
    } else {
        for (int r = tid; r < R; r += SEL_THREADS) {
            long long above = 0, ln;
            if (in_lds) {
                const RunRec me = s_run[r];
                ln = me.len;
                // eight records read before they are compared: one LDS round
                // trip per eight runs rather than per run
                int r2 = 0;
                for (; r2 + 8 <= R; r2 += 8) {
                    RunRec o[8];
#pragma unroll
                    for (int q = 0; q < 8; ++q) o[q] = s_run[r2 + q];
#pragma unroll
                    for (int q = 0; q < 8; ++q)
                        if (o[q].bkt == me.bkt && o[q].key > me.key) above += o[q].len;
                }
                for (; r2 < R; ++r2) {
                    const RunRec o = s_run[r2];
                    if (o.bkt == me.bkt && o.key > me.key) above += o.len;
                }
            } else {
                const unsigned long long key = a.run_key[r];
                const int bk = a.run_bkt[r];
                ln = a.run_start[r + 1] - a.run_start[r];
                for (int r2 = 0; r2 < R; ++r2)
                    if (a.run_bkt[r2] == bk && a.run_key[r2] > key) above += a.run_start[r2 + 1] - a.run_start[r2];
            }
            const long long t = min(ln, max(0LL, quota - above));
            a.run_take[r] = (int)t;
            if (in_lds) s_take[r] = (int)t;
            taken += t;
        }
    }
    taken = block_sum_ll(taken, s_ll);
    const long long fill = (long long)(a.M - a.n_s - a.n_w) - taken;
    // beyond RUN_CAP runs the fill pass below reads run_take of runs that other
    // waves stored to global memory: a full barrier (workgroup-scope release and
    // acquire of global memory) orders those stores before the reads; the
    // barriers inside block_sum_ll fence LDS only
    __syncthreads();

    // ---- fill with the best remaining tokens over all spans; a run keeps
    // its newest tokens, slots [run_from, run end)
    if (by_sort) {
        sort_runs([&](int x, int y) {  // key descending
            if (x >= R) return false;
            if (y >= R) return true;
            return s_run[x].key > s_run[y].key;
        });
        const int r0 = i0 < R ? s_ord[i0] : -1, r1 = i1 < R ? s_ord[i1] : -1;
        const int t0 = r0 >= 0 ? s_take[r0] : 0, t1 = r1 >= 0 ? s_take[r1] : 0;
        const int m0 = r0 >= 0 ? s_run[r0].len - t0 : 0, m1 = r1 >= 0 ? s_run[r1].len - t1 : 0;
        const int f0 = block_excl_scan(m0 + m1, s_scan, tot), f1 = f0 + m0;  // left in better runs
        if (r0 >= 0) {
            const int from = a.run_start[r0 + 1] - (t0 + (int)min((long long)m0, max(0LL, fill - f0)));
            a.run_from[r0] = from;
            s_from[r0] = from;
        }
        if (r1 >= 0) {
            const int from = a.run_start[r1 + 1] - (t1 + (int)min((long long)m1, max(0LL, fill - f1)));
            a.run_from[r1] = from;
            s_from[r1] = from;
        }
    } else {
        for (int r = tid; r < R; r += SEL_THREADS) {
            long long above = 0, ln, tk;
            if (in_lds) {
                const RunRec me = s_run[r];
                ln = me.len;
                tk = s_take[r];
                int r2 = 0;
                for (; r2 + 8 <= R; r2 += 8) {
                    RunRec o[8];
                    int tq[8];
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        o[q] = s_run[r2 + q];
                        tq[q] = s_take[r2 + q];
                    }
#pragma unroll
                    for (int q = 0; q < 8; ++q)
                        if (o[q].key > me.key) above += o[q].len - tq[q];
                }
                for (; r2 < R; ++r2) {
                    const RunRec o = s_run[r2];
                    if (o.key > me.key) above += o.len - s_take[r2];
                }
            } else {
                const unsigned long long key = a.run_key[r];
                ln = a.run_start[r + 1] - a.run_start[r];
                tk = a.run_take[r];
                for (int r2 = 0; r2 < R; ++r2)
                    if (a.run_key[r2] > key) above += (a.run_start[r2 + 1] - a.run_start[r2]) - a.run_take[r2];
            }
            const long long f = min(ln - tk, max(0LL, fill - above));
            const int from = a.run_start[r + 1] - (int)(tk + f);
            a.run_from[r] = from;
            if (in_lds) s_from[r] = from;
        }
    }
    __syncthreads();
    auto run_from = [&](int r) { return in_lds ? s_from[r] : a.run_from[r]; };

    // ---- pass 2: keep list (ascending) and its inverse on destinations [0, M)
    int total_kept = 0;
    int first_move = a.M;  // smallest destination d with keep[d] != d
    int split = a.M;       // smallest destination d with keep[d] - d >= stage_shift
    const int n_evict = a.len - a.M;
    // the next block's entries are loaded while this one is processed
    int n2ch[SEL_PER], n2sl[SEL_PER], n2pc = -1, n2r = -1;
    auto fetch2 = [&](int base) {
        const int lo = base + tid * SEL_PER;
        load_block(a.chunk, lo, a.len, n2ch);
        if (a.slot) load_block(a.slot, lo, a.len, n2sl);
        n2pc = (lo > 0 && lo <= a.len) ? a.chunk[lo - 1] : -1;
        n2r = (lo < a.len) ? a.th_run[base / SEL_PER + tid] - 1 : -1;  // run holding the slot before lo
    };
    if (a.len > 0) fetch2(0);
    for (int base = 0; base < a.len; base += SEL_BLOCK) {
        const int lo = base + tid * SEL_PER;
        int ch[SEL_PER], sl[SEL_PER];
#pragma unroll
        for (int k = 0; k < SEL_PER; ++k) {
            ch[k] = n2ch[k];
            sl[k] = n2sl[k];
        }
        int pc = n2pc;
        int r = n2r;
        if (base + SEL_BLOCK < a.len) fetch2(base + SEL_BLOCK);
        int from = (r >= 0 && r < R) ? run_from(r) : 0;
        unsigned mask = 0;
#pragma unroll
        for (int k = 0; k < SEL_PER; ++k) {
            const int i = lo + k;
            if (i < a.len) {
                bool kept = true;
                if (i >= c0 && i < c1) {
                    if (i == c0 || ch[k] != pc) {
                        ++r;
                        from = run_from(r);
                    }
                    kept = i >= from;
                }
                if (kept) mask |= 1u << k;
                pc = ch[k];
            }
        }
        // the block's keep entries and freed slots are collected in LDS and
        // leave as contiguous stores; the inverse leaves as one 16-byte store
        // per thread (scattered 4-byte stores would load the memory pipeline)
        int tot = 0;
        int off = total_kept + block_excl_scan(__popc(mask), s_scan, tot);
        const int ev_base = base - total_kept;  // tokens evicted before this block
        int invv[SEL_PER];
#pragma unroll
        for (int k = 0; k < SEL_PER; ++k) {
            const int i = lo + k;
            invv[k] = -1;
            if (i < a.len) {
                if (mask & (1u << k)) {
                    if (off < a.M) {
                        s_keep[off - total_kept] = i;
                        if (off != i) first_move = min(first_move, off);
                        if (i - off >= a.stage_shift) split = min(split, off);
                    }
                    invv[k] = off;
                    ++off;
                } else if (a.slot) {
                    // evicted token i is the (i - off)-th evicted one in logical order
                    s_free[i - off - ev_base] = sl[k];
                }
            }
        }
        if (lo + SEL_PER <= a.M) {
            *(int4 *)(a.inv + lo) = int4{invv[0], invv[1], invv[2], invv[3]};
        } else {
#pragma unroll
            for (int k = 0; k < SEL_PER; ++k)
                if (lo + k < a.M) a.inv[lo + k] = invv[k];
        }
        lds_sync();
        const int kn = min(tot, a.M - total_kept);
        for (int q = tid; q < kn; q += SEL_THREADS) {
            a.keep[total_kept + q] = s_keep[q];
            if (a.keep_out) a.keep_out[total_kept + q] = s_keep[q];
        }
        if (a.slot) {
            const int fn = min(min(a.len - base, SEL_BLOCK) - tot, n_evict - ev_base);
            for (int q = tid; q < fn; q += SEL_THREADS) a.free_out[ev_base + q] = s_free[q];
        }
        lds_sync();
        total_kept += tot;
    }
    // ---- moving destinations form the suffix [first_move, M) (keep[d] - d is
    // nondecreasing); clear their flags for the gather
    {
        // minimum over the block: within each wave by lane exchanges, then over
        // the 16 wave results (one LDS atomic per thread would serialize)
        __shared__ int s_first[SEL_THREADS / 64], s_split[SEL_THREADS / 64];
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) {
            first_move = min(first_move, __shfl_xor(first_move, off, 64));
            split = min(split, __shfl_xor(split, off, 64));
        }
        if ((tid & 63) == 0) {
            s_first[tid >> 6] = first_move;
            s_split[tid >> 6] = split;
        }
        lds_sync();
#pragma unroll
        for (int w = 0; w < SEL_THREADS / 64; ++w) {
            first_move = min(first_move, s_first[w]);
            split = min(split, s_split[w]);
        }
        split = max(split, first_move);
    }
    if (tid == 0) {
        a.status[3] = first_move;
        a.status[4] = split;
        const bool count_ok = total_kept == a.M;
        if (!count_ok) {  // cannot happen for valid arguments; never move data then
            a.status[0] = 2;
            a.status[1] = 1;
        }
        if (a.outcome_out) *a.outcome_out = count_ok ? 0 : 2;
    }
    {
        // flags of the moving destinations back to zero, 16 bytes per store
        const int fs = first_move * a.n_chunks, fe = a.n_flags;
        const int fa = min((fs + 3) & ~3, fe), fb = max(fa, fe & ~3);
        if (tid < fa - fs) a.flags[fs + tid] = 0;
        for (int q = fa / 4 + tid; q < fb / 4; q += SEL_THREADS) ((int4 *)a.flags)[q] = int4{0, 0, 0, 0};
        if (tid < fe - fb) a.flags[fb + tid] = 0;
    }

    // ---- indexed variant: pos, chunk_id and slot move down in place,
    // new[d] = old[keep[d]] for the moving destinations [first_move, M).
    // keep[d] >= d, so a block of destinations only reads at or above its own
    // start; each block reads everything before any thread writes, and the
    // next block's reads lie above what this block writes.
    if (a.slot && total_kept == a.M) {
        __syncthreads();  // the keep list written above by every thread is read below
        // the keep entries of the next block are loaded while this block moves
        // (the pass never writes the keep list): one dependent round trip to
        // memory per block instead of two
        int nk[SEL_PER];
        auto fetch_keep = [&](int base) __attribute__((always_inline)) {
#pragma unroll
            for (int k = 0; k < SEL_PER; ++k) {
                const int d = base + k * SEL_THREADS + tid;
                nk[k] = d < a.M ? a.keep[d] : 0;
            }
        };
        if (first_move < a.M) fetch_keep(first_move);
        for (int base = first_move; base < a.M; base += SEL_BLOCK) {
            int vp[SEL_PER], vc[SEL_PER], vs[SEL_PER], kk[SEL_PER];
#pragma unroll
            for (int k = 0; k < SEL_PER; ++k) kk[k] = nk[k];
            if (base + SEL_BLOCK < a.M) fetch_keep(base + SEL_BLOCK);
#pragma unroll
            for (int k = 0; k < SEL_PER; ++k) {
                const int d = base + k * SEL_THREADS + tid;
                if (d < a.M) {
                    const int src = kk[k];
                    vp[k] = a.pos[src];
                    vc[k] = a.chunk[src];
                    vs[k] = a.slot[src];
                }
            }
            __syncthreads();
#pragma unroll
            for (int k = 0; k < SEL_PER; ++k) {
                const int d = base + k * SEL_THREADS + tid;
                if (d < a.M) {
                    a.pos[d] = vp[k];
                    a.chunk[d] = vc[k];
                    a.slot[d] = vs[k];
                }
            }
        }
    }
}

struct GatherArgs {
    char *const *plane_tab;
    uint32_t row_bytes, row_units;  // bytes and 16-byte units of one plane row
    int n_planes, planes_per_group;
    int M, n_chunks;
    int32_t *pos, *chunk;
    const int32_t *keep, *inv;
    int32_t *flags, *status;
    uint32_t *ticket;
    char *trash;  // 8 KiB that stores with nothing to write go to (the staging area, idle by then)
};

// s_waitcnt immediate that waits until at most n vector memory operations of
// this wave are in flight (lgkm and exp counters not waited for)
constexpr int vmcnt_imm(int n) { return 0x0F70 | (n & 15) | ((n >> 4) << 14); }

// Moving destinations [first, M) are handed out in ticket order, ROWS
// consecutive slots per ticket; for each slot and each group of planes the
// workgroup reads the source rows, signals, waits for the reader of the slot
// and writes.  KPR = 16-byte units per thread per plane row
// (row_bytes <= 4096 KPR); a plane group holds 16 / KPR plane rows.
constexpr int GATHER_ROWS = 8;
// workgroups of the gather, each taking tickets until none is left: three for
// every four CUs of MI355X moved a 1 GiB eviction fastest (fewer streams of
// copies in flight than one per CU, which also beat one per ticket)
constexpr int GATHER_WG = 192;

template <int KPR>
__global__ __launch_bounds__(256) void kv_gather_kernel(GatherArgs a) {
    constexpr int PPG = GATHER_U / KPR;
    __shared__ int s_t;
    __shared__ int s_src[GATHER_ROWS], s_dep[GATHER_ROWS];
    __shared__ char *s_pt[KV_MAX_PLANES];
    if (a.status[1]) return;
    const int first = a.status[4];
    const int n_work = (a.M - first + GATHER_ROWS - 1) / GATHER_ROWS;
    if ((int)blockIdx.x >= n_work) return;  // more workgroups than moving rows: take no ticket
    const int tid = threadIdx.x;
    if (tid < a.n_planes) s_pt[tid] = a.plane_tab[tid];
    // tickets are taken until none is left, so the grid drains evenly; a
    // workgroup only waits for slots of lower tickets, which running
    // workgroups hold
    __shared__ int s_stop;
    for (;;) {
        if (tid == 0) {
            s_t = (int)atomicAdd(a.ticket, 1u);
            // a workgroup whose wait timed out stopped every move: take no more work
            s_stop = __hip_atomic_load(&a.status[1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        __syncthreads();
        if (s_t >= n_work || s_stop) break;
        const int d_lo = first + s_t * GATHER_ROWS;
        const int d_hi = min(d_lo + GATHER_ROWS, a.M);
        // sources and readers of the ticket's slots, in LDS: a global load inside
        // the pipeline below would make the compiler wait for every load in flight
        if (tid < d_hi - d_lo) {
            s_src[tid] = a.keep[d_lo + tid];
            s_dep[tid] = a.inv[d_lo + tid];  // destination whose source is row d (-1 if row d is evicted)
        }
        __syncthreads();

        // Units u = (slot d_lo + u / n_chunks, plane group u % n_chunks) in two
        // register buffers.  Per unit: wait for its loads, signal that its source
        // rows are held, wait for the reader of its slot, issue the next unit's
        // loads, write the slot -- so a workgroup's writes overlap its next reads.
        // Each unit issues exactly LPU loads and LPU stores per lane (lanes with
        // nothing to store write to the trash area) so that the wait can count them
        // (vmcnt counts loads and stores together, in issue order); plane pointers
        // and slot metadata come from LDS, since a global load whose value is used
        // at once would make the compiler wait for every load in flight.
        constexpr int LPU = GATHER_U + 2;
        const int n_units = (d_hi - d_lo) * a.n_chunks;
        u32x4 bufA[GATHER_U], bufB[GATHER_U];
        int pvA = 0, cvA = 0, pvB = 0, cvB = 0;
        auto load = [&](int u, u32x4 (&buf)[GATHER_U], int &pv, int &cv) __attribute__((always_inline)) {
            const int c = u % a.n_chunks;
            const int src = s_src[u / a.n_chunks];
            const int p0 = c * a.planes_per_group;
            // (units past the row or planes past the group re-read a valid address)
    #pragma clang loop unroll(full)
            for (int pi = 0; pi < PPG; ++pi) {
                const int p = min(p0 + pi, a.n_planes - 1);
                GPTR(const char) row = (GPTR(const char))s_pt[p] + (size_t)src * a.row_bytes;
    #pragma clang loop unroll(full)
                for (int k = 0; k < KPR; ++k) {
                    const uint32_t unit = min((uint32_t)(tid + 256 * k), a.row_units - 1);
                    buf[pi * KPR + k] = *(GPTR(const u32x4))(row + 16u * unit);
                }
            }
            pv = a.pos[src];  // position and chunk id of the source row (lane 0 of group 0 stores them)
            cv = a.chunk[src];
        };
        auto step = [&](int u, const u32x4 (&buf)[GATHER_U], int pv, int cv, u32x4 (&nbuf)[GATHER_U], int &npv, int &ncv)
            __attribute__((always_inline)) {
            const int d = d_lo + u / a.n_chunks, c = u % a.n_chunks;
            const int dep = s_dep[u / a.n_chunks];
            // this unit's loads: after them only the previous unit's stores were issued
            if (u == 0)
                __builtin_amdgcn_s_waitcnt(vmcnt_imm(0));
            else
                __builtin_amdgcn_s_waitcnt(vmcnt_imm(LPU));
            lds_sync();  // every lane holds this unit's source rows
            if (tid == 0) {
                __hip_atomic_store(&a.flags[d * a.n_chunks + c], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                // ---- wait until the reader of row d (a lower slot, hence an
                // earlier ticket or an earlier unit here) holds its data.  The
                // wait is bounded: on a timeout every move stops (status[1]) and
                // the call's outcome becomes 3; a workgroup that sees the stop
                // while waiting leaves as well, without writing
                if (dep >= first && dep != d) {  // readers below `first` were staged earlier
                    int it = 0;
                    const int ft = dep * a.n_chunks + c;
                    while (__hip_atomic_load(&a.flags[ft], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
                        if (++it >= SPIN_LIMIT) {
                            __hip_atomic_store(&a.status[2], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                            __hip_atomic_store(&a.status[0], 3, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                            __hip_atomic_store(&a.status[1], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                            s_stop = 1;
                            break;
                        }
                        if ((it & 63) == 0 &&
                            __hip_atomic_load(&a.status[1], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
                            s_stop = 1;
                            break;
                        }
                        __builtin_amdgcn_s_sleep(2);
                    }
                }
            }
            lds_sync();
            if (s_stop) return false;
            load(min(u + 1, n_units - 1), nbuf, npv, ncv);  // unconditional (a repeat past the end is never written)
            // ---- write slot d
            const int p0 = c * a.planes_per_group;
            GPTR(u32x4) trash = (GPTR(u32x4))a.trash + tid;
    #pragma clang loop unroll(full)
            for (int pi = 0; pi < PPG; ++pi) {
                const int p = p0 + pi;
                const bool plane_ok = pi < a.planes_per_group && p < a.n_planes;
                GPTR(char) row = (GPTR(char))s_pt[min(p, a.n_planes - 1)] + (size_t)d * a.row_bytes;
    #pragma clang loop unroll(full)
                for (int k = 0; k < KPR; ++k) {
                    const uint32_t unit = (uint32_t)(tid + 256 * k);
                    GPTR(u32x4) dst = (plane_ok && unit < a.row_units) ? (GPTR(u32x4))(row + 16u * unit) : trash;
                    __builtin_nontemporal_store(buf[pi * KPR + k], dst);  // streaming: 230 -> 218 us on a 1 GiB event
                }
            }
            const bool meta = c == 0 && tid == 0;
            int32_t *tr = (int32_t *)(a.trash + 4096) + 2 * tid;
            *(meta ? a.pos + d : tr) = pv;
            *(meta ? a.chunk + d : tr + 1) = cv;
            return true;
        };
        load(0, bufA, pvA, cvA);
        for (int u = 0; u < n_units; u += 2) {
            if (!step(u, bufA, pvA, cvA, bufB, pvB, cvB)) return;  // moves stopped (s_stop is workgroup-uniform)
            if (u + 1 < n_units && !step(u + 1, bufB, pvB, cvB, bufA, pvA, cvA)) return;
        }
        __syncthreads();  // every lane is done with this ticket's LDS entries
    }
}

struct StageArgs {
    char *const *plane_tab;
    uint32_t row_bytes, row_units;
    int n_planes, planes_per_group, n_chunks;
    int rows, block;  // destinations [block * rows, (block + 1) * rows)
    int32_t *pos, *chunk;
    const int32_t *keep, *status;
    char *area;       // [rows][n_chunks][256 threads][16 units] 16-byte units
    int32_t *meta;    // [rows][2] positions and chunk ids
};

template <int KPR, bool READ>
__device__ __forceinline__ void kv_stage_row(const StageArgs &a, int r, int c) {
    constexpr int PPG = GATHER_U / KPR;
    const int tid = threadIdx.x;
    const int d = a.block * a.rows + r;
    GPTR(u32x4) slot = (GPTR(u32x4))(a.area + ((size_t)r * a.n_chunks + c) * (size_t)(GATHER_U * 16 * 256));
    const int row = READ ? a.keep[d] : d;
    const int p0 = c * a.planes_per_group;
#pragma clang loop unroll(full)
    for (int pi = 0; pi < PPG; ++pi) {
        const int p = p0 + pi;
        if (pi >= a.planes_per_group || p >= a.n_planes) break;
        GPTR(char) base = (GPTR(char))a.plane_tab[p] + (size_t)row * a.row_bytes;
#pragma clang loop unroll(full)
        for (int k = 0; k < KPR; ++k) {
            const uint32_t unit = (uint32_t)(tid + 256 * k);
            if (unit < a.row_units) {
                GPTR(u32x4) g = (GPTR(u32x4))(base + 16u * unit);
                GPTR(u32x4) t = slot + (pi * KPR + k) * 256 + tid;
                // nontemporal stores, as in the ticket gather (streamed chunks ~1 % faster)
                if (READ) __builtin_nontemporal_store(*g, t); else __builtin_nontemporal_store(*t, g);
            }
        }
    }
    if (c == 0 && tid == 0) {
        if (READ) {
            a.meta[2 * r] = a.pos[row];
            a.meta[2 * r + 1] = a.chunk[row];
        } else {
            a.pos[d] = a.meta[2 * r];
            a.chunk[d] = a.meta[2 * r + 1];
        }
    }
}

// Workgroup x of plane group y handles destinations x, x + STAGE_WG, ... of
// the block.  READ copies the source rows of the staged destinations into the
// area, WRITE copies them to their slots.  Destinations outside
// [status[3], status[4]) are skipped, so a launch with nothing to stage ends
// at once.
template <int KPR, bool READ>
__global__ __launch_bounds__(256) void kv_stage_kernel(StageArgs a) {
    if (a.status[1]) return;
    const int lo = max(a.status[3] - a.block * a.rows, 0);
    const int hi = min(a.status[4] - a.block * a.rows, a.rows);
    for (int r = lo + (int)blockIdx.x; r < hi; r += (int)gridDim.x) kv_stage_row<KPR, READ>(a, r, (int)blockIdx.y);
}

// 16-byte units per thread per plane row, rounded up to a power of two.
static int gather_kpr(int row_bytes) {
    const int need = (row_bytes + 4095) / 4096;
    int k = 1;
    while (k < need) k *= 2;
    return k;
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Scratch of the indexed eviction for callers that cannot allocate: one copy
// per GPU, held until the process ends.  Host code never passes the array's
// name to a kernel (on the host it is a stand-in, not a device address); it
// passes the address hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) char scratch[KV_NOALLOC_SCRATCH_BYTES];

hipError_t kv_noalloc_scratch(char **out) {
    constexpr int MAX_DEV = 64;
    static std::mutex mu;
    static char *addr[MAX_DEV] = {};
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= MAX_DEV) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        addr[dev] = (char *)p;
    }
    *out = addr[dev];
    return hipSuccess;
}

KvWorkspace kv_workspace_layout(int n_layers, int row_bytes, int capacity) {
    KvWorkspace w{};
    const int ppg = GATHER_U / gather_kpr(row_bytes);
    w.n_chunks = (2 * n_layers + ppg - 1) / ppg;
    const size_t cap = (size_t)capacity;
    const size_t blocks = (cap + SEL_BLOCK - 1) / SEL_BLOCK;
    size_t off = 0;
    w.offStatus = off;
    off = align256(off + 64);
    w.offPlanes = off;
    off = align256(off + KV_MAX_PLANES * sizeof(char *));
    w.offKeep = off;
    off = align256(off + cap * 4);
    w.offInv = off;
    off = align256(off + cap * 4);
    w.offThRun = off;
    off = align256(off + blocks * SEL_THREADS * 4);
    w.offRunStart = off;
    off = align256(off + (cap + 1) * 4);
    w.offRunKey = off;
    off = align256(off + cap * 8);
    w.offRunBkt = off;
    off = align256(off + cap * 4);
    w.offRunTake = off;
    off = align256(off + cap * 4);
    w.offRunFrom = off;
    off = align256(off + cap * 4);
    w.offFlags = off;
    off = align256(off + cap * (size_t)w.n_chunks * 4);
    w.stage_rows = 0;
    w.offStage = w.offStageMeta = off;
    if (w.n_chunks > 0) {
        const long long per_row = (long long)w.n_chunks * GATHER_U * 16 * 256;
        w.stage_rows = (int)std::max(1ll, std::min((long long)capacity, STAGE_AREA / per_row));
        w.offStage = off;
        off = align256(off + (size_t)w.stage_rows * per_row);
        w.offStageMeta = off;
        off = align256(off + (size_t)w.stage_rows * 8);
    }
    w.total = off;
    return w;
}

// ---------------------------------------------------------------------------
// kv_append_indexed: workgroup (t, p) for t < T copies row t of plane p's new
// rows into row s_t of the plane, s_t the t-th entry of the free list
// free_a ++ free_b, 16 bytes a thread; the workgroups of plane 0 also write the
// token's pos, chunk id and slot; workgroups past T (plane 0) copy the rest of
// the free list to free_rest.  Entries outside [0, capacity) are skipped.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void kv_append_kernel(KvAppendLaunch a) {
    const int t = blockIdx.x, p = blockIdx.y;
    auto free_at = [&](int i) { return i < a.na ? a.free_a[i] : a.free_b[i - a.na]; };
    if (t < a.T) {
        const int s = free_at(t);
        if (s < 0 || s >= a.capacity) return;
        const uint4 *src = (const uint4 *)(a.new_rows[p] + (size_t)t * a.row_bytes);
        uint4 *dst = (uint4 *)(a.planes[p] + (size_t)s * a.row_bytes);
        for (int i = threadIdx.x; i < a.row_bytes / 16; i += 256) dst[i] = src[i];
        if (p == 0 && threadIdx.x == 0) {
            a.pos[a.n + t] = a.pos0 + t;
            a.chunk_id[a.n + t] = a.chunk;
            a.slot[a.n + t] = s;
        }
    } else if (p == 0) {
        const int i = (t - a.T) * 256 + threadIdx.x;  // index into the rest of the list
        if (i < a.na + a.nb - a.T) a.free_rest[i] = free_at(a.T + i);
    }
}

hipError_t launch_kv_append(const KvAppendLaunch &p, hipStream_t stream) {
    const int rest = p.na + p.nb - p.T;
    const int gx = p.T + (rest + 255) / 256;
    if (gx == 0) return hipSuccess;
    hipLaunchKernelGGL(kv_append_kernel, dim3(gx, p.n_planes), dim3(256), 0, stream, p);
    return hipGetLastError();
}

hipError_t launch_kv_evict(const KvLaunch &p, hipStream_t stream) {
    char *ws = p.ws;
    KvArgs a;
    a.pos = p.pos;
    a.chunk = p.chunk_id;
    a.scores = p.chunk_scores;
    a.num_chunks = p.num_chunks;
    a.len = p.len;
    a.M = p.M;
    a.n_s = p.n_sink;
    a.n_w = p.n_window;
    a.N = p.n_buckets;
    a.n_flags = p.M * p.lay.n_chunks;
    a.n_chunks = p.lay.n_chunks;
    {
        // stage destinations whose shift spans less than STAGE_BYTES of rows
        const long long row_all = (long long)std::max(p.n_planes, 1) * p.row_bytes;
        a.stage_shift = (int)std::min((long long)p.M + 1, (STAGE_BYTES + row_all - 1) / row_all);
        if (p.slot) a.stage_shift = p.M + 1;  // the indexed variant moves no rows
    }
    a.status = (int32_t *)(ws + p.lay.offStatus);
    a.ticket = (uint32_t *)(ws + p.lay.offStatus + 32);
    a.keep = (int32_t *)(ws + p.lay.offKeep);
    a.inv = (int32_t *)(ws + p.lay.offInv);
    a.th_run = (int32_t *)(ws + p.lay.offThRun);
    a.run_start = (int32_t *)(ws + p.lay.offRunStart);
    a.run_key = (unsigned long long *)(ws + p.lay.offRunKey);
    a.run_bkt = (int32_t *)(ws + p.lay.offRunBkt);
    a.run_take = (int32_t *)(ws + p.lay.offRunTake);
    a.run_from = (int32_t *)(ws + p.lay.offRunFrom);
    a.flags = (int32_t *)(ws + p.lay.offFlags);
    a.keep_out = p.keep_out;
    a.slot = p.slot;
    a.free_out = p.free_out;
    a.outcome_out = p.outcome_out;
    a.plane_tab = (char **)(ws + p.lay.offPlanes);
    for (int i = 0; i < KV_MAX_PLANES; ++i) a.planes[i] = i < p.n_planes ? p.planes[i] : nullptr;
    a.n_planes = p.n_planes;
    hipLaunchKernelGGL(kv_select_kernel, dim3(1), dim3(SEL_THREADS), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || p.slot) return e;  // the indexed variant moves no rows

    const long long groups = (long long)p.M * p.lay.n_chunks;
    if (groups == 0) return hipSuccess;
    GatherArgs g;
    const int kpr = gather_kpr(p.row_bytes);
    g.plane_tab = a.plane_tab;
    g.row_bytes = (uint32_t)p.row_bytes;
    g.row_units = (uint32_t)(p.row_bytes / 16);
    g.n_planes = p.n_planes;
    g.planes_per_group = GATHER_U / kpr;
    g.trash = ws + p.lay.offStage;
    g.M = p.M;
    g.n_chunks = p.lay.n_chunks;
    g.pos = p.pos;
    g.chunk = p.chunk_id;
    g.keep = a.keep;
    g.inv = a.inv;
    g.flags = a.flags;
    g.status = a.status;
    g.ticket = a.ticket;
    // staged destinations first (block by block, in order), then the ticket gather
    StageArgs sa;
    sa.plane_tab = a.plane_tab;
    sa.row_bytes = g.row_bytes;
    sa.row_units = g.row_units;
    sa.n_planes = p.n_planes;
    sa.planes_per_group = g.planes_per_group;
    sa.n_chunks = p.lay.n_chunks;
    sa.rows = p.lay.stage_rows;
    sa.pos = p.pos;
    sa.chunk = p.chunk_id;
    sa.keep = a.keep;
    sa.status = a.status;
    sa.area = p.ws + p.lay.offStage;
    sa.meta = (int32_t *)(p.ws + p.lay.offStageMeta);
    const dim3 sgrid((unsigned)std::min(sa.rows, STAGE_WG), (unsigned)sa.n_chunks), blk(256);
    for (int b = 0; (long long)b * sa.rows < p.M; ++b) {
        sa.block = b;
        switch (kpr) {
        case 1:
            hipLaunchKernelGGL((kv_stage_kernel<1, true>), sgrid, blk, 0, stream, sa);
            hipLaunchKernelGGL((kv_stage_kernel<1, false>), sgrid, blk, 0, stream, sa);
            break;
        case 2:
            hipLaunchKernelGGL((kv_stage_kernel<2, true>), sgrid, blk, 0, stream, sa);
            hipLaunchKernelGGL((kv_stage_kernel<2, false>), sgrid, blk, 0, stream, sa);
            break;
        case 4:
            hipLaunchKernelGGL((kv_stage_kernel<4, true>), sgrid, blk, 0, stream, sa);
            hipLaunchKernelGGL((kv_stage_kernel<4, false>), sgrid, blk, 0, stream, sa);
            break;
        case 8:
            hipLaunchKernelGGL((kv_stage_kernel<8, true>), sgrid, blk, 0, stream, sa);
            hipLaunchKernelGGL((kv_stage_kernel<8, false>), sgrid, blk, 0, stream, sa);
            break;
        default:
            hipLaunchKernelGGL((kv_stage_kernel<16, true>), sgrid, blk, 0, stream, sa);
            hipLaunchKernelGGL((kv_stage_kernel<16, false>), sgrid, blk, 0, stream, sa);
            break;
        }
        e = hipGetLastError();
        if (e != hipSuccess) return e;
    }
    const dim3 grid((unsigned)std::min((p.M + GATHER_ROWS - 1) / GATHER_ROWS, GATHER_WG));
    switch (kpr) {
    case 1: hipLaunchKernelGGL(kv_gather_kernel<1>, grid, blk, 0, stream, g); break;
    case 2: hipLaunchKernelGGL(kv_gather_kernel<2>, grid, blk, 0, stream, g); break;
    case 4: hipLaunchKernelGGL(kv_gather_kernel<4>, grid, blk, 0, stream, g); break;
    case 8: hipLaunchKernelGGL(kv_gather_kernel<8>, grid, blk, 0, stream, g); break;
    default: hipLaunchKernelGGL(kv_gather_kernel<16>, grid, blk, 0, stream, g); break;
    }
    return hipGetLastError();
}

}  // namespace ds
