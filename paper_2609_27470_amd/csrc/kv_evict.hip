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
//   * kept slots -> ascending keep list, its inverse on [0, M), and a
//     per-destination flag array for the gather.
// kv_gather moves the kept rows down in place.  Slot d receives row keep[d]
// (keep[d] >= d).  Writing slot d is safe once the reader of row d -- the
// destination inv[d] < d, if row d is kept -- has its data in registers.
// Workgroups take increasing tickets, signal "read done" before they wait,
// and only ever wait on lower tickets, so every wait ends; the wait is also
// bounded and reports a timeout in the status word instead of hanging.
#include "common.h"
#include "kernels.h"

namespace ds {

constexpr int SEL_THREADS = 1024;
constexpr int GATHER_U = 16;                        // uint4 per thread per group
constexpr int GATHER_BYTES = 256 * 16 * GATHER_U;   // 64 KiB per group
constexpr int SPIN_LIMIT = 1 << 22;

struct KvArgs {
    const int32_t *pos_in;
    const int32_t *chunk;
    const float *scores;
    int num_chunks, len, M, n_s, n_w, N;
    int n_flags;
    int32_t *status;   // [0] invariants broken, [1] skip gather, [2] wait timed out
    uint32_t *ticket;
    int32_t *keep, *inv, *mask, *run_start, *run_bkt, *run_take;
    unsigned long long *run_key;
    int32_t *flags;
    int32_t *keep_out;
};

__device__ __forceinline__ uint32_t orderable(float f) {
    const uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Exclusive prefix sum over the 1024 threads of the block.
__device__ int block_excl_scan(int x, int *s_tmp, int &total) {
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
    int incl = x;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
        const int y = __shfl_up(incl, off, 64);
        if (lane >= off) incl += y;
    }
    if (lane == 63) s_tmp[wid] = incl;
    __syncthreads();
    if (tid == 0) {
        int acc = 0;
        for (int i = 0; i < SEL_THREADS / 64; ++i) {
            const int t = s_tmp[i];
            s_tmp[i] = acc;
            acc += t;
        }
        s_tmp[SEL_THREADS / 64] = acc;
    }
    __syncthreads();
    const int res = s_tmp[wid] + incl - x;
    total = s_tmp[SEL_THREADS / 64];
    __syncthreads();
    return res;
}

__device__ long long block_sum_ll(long long x, long long *s_tmp) {
    const int tid = threadIdx.x, lane = tid & 63, wid = tid >> 6;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, 64);
    if (lane == 0) s_tmp[wid] = x;
    __syncthreads();
    if (tid == 0) {
        long long acc = 0;
        for (int i = 0; i < SEL_THREADS / 64; ++i) acc += s_tmp[i];
        s_tmp[SEL_THREADS / 64] = acc;
    }
    __syncthreads();
    const long long r = s_tmp[SEL_THREADS / 64];
    __syncthreads();
    return r;
}

__global__ __launch_bounds__(SEL_THREADS) void kv_select_kernel(KvArgs a) {
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
    for (int i = tid; i < a.n_flags; i += SEL_THREADS) a.flags[i] = 0;
    __syncthreads();

    // ---- cache invariants: chunk ids in range and nondecreasing, positions increasing
    {
        int bad = 0;
        for (int i = tid; i < a.len; i += SEL_THREADS) {
            const int c = a.chunk[i];
            if (c < 0 || c >= a.num_chunks) bad = 1;
            if (i > 0 && (c < a.chunk[i - 1] || a.pos_in[i] <= a.pos_in[i - 1])) bad = 1;
        }
        if (bad) atomicOr(&s_bad, 1);
    }
    __syncthreads();
    if (s_bad) {
        if (tid == 0) {
            a.status[0] = 1;
            a.status[1] = 1;
        }
        return;
    }

    // ---- runs of equal chunk id among the candidates [c0, c1)
    const int c0 = a.n_s, c1 = a.len - a.n_w, ncand = c1 - c0;
    int R = 0;
    {
        const int per = (ncand + SEL_THREADS - 1) / SEL_THREADS;
        const int lo = c0 + tid * per, hi = min(lo + per, c1);
        int cnt = 0;
        for (int i = lo; i < hi; ++i) cnt += (i == c0 || a.chunk[i] != a.chunk[i - 1]);
        int off = block_excl_scan(cnt, s_scan, R);
        for (int i = lo; i < hi; ++i)
            if (i == c0 || a.chunk[i] != a.chunk[i - 1]) a.run_start[off++] = i;
        if (tid == 0) a.run_start[R] = c1;
    }
    __syncthreads();

    const int a_min = (ncand > 0) ? a.chunk[c0] : 0;
    const int a_max = (ncand > 0) ? a.chunk[c1 - 1] : 0;
    const long long span = (long long)a_max - a_min + 1;
    const int N = max(1, a.N);
    for (int r = tid; r < R; r += SEL_THREADS) {
        const int ch = a.chunk[a.run_start[r]];
        a.run_key[r] = ((unsigned long long)orderable(a.scores[ch]) << 32) | (unsigned)ch;
        a.run_bkt[r] = (int)(((long long)N * (ch - a_min)) / span);
    }
    __syncthreads();

    // ---- per-span quota: a run keeps what the better runs of its span left
    const long long quota = (a.M - a.n_s - a.n_w) / N;
    long long taken = 0;
    for (int r = tid; r < R; r += SEL_THREADS) {
        const unsigned long long key = a.run_key[r];
        const int bk = a.run_bkt[r];
        const long long ln = a.run_start[r + 1] - a.run_start[r];
        long long above = 0;
        for (int r2 = 0; r2 < R; ++r2)
            if (a.run_bkt[r2] == bk && a.run_key[r2] > key) above += a.run_start[r2 + 1] - a.run_start[r2];
        const long long t = min(ln, max(0LL, quota - above));
        a.run_take[r] = (int)t;
        taken += t;
    }
    taken = block_sum_ll(taken, s_ll);
    const long long fill = (long long)(a.M - a.n_s - a.n_w) - taken;

    // ---- fill: best remaining tokens over all spans
    for (int r = tid; r < R; r += SEL_THREADS) {
        const unsigned long long key = a.run_key[r];
        const long long left = (a.run_start[r + 1] - a.run_start[r]) - a.run_take[r];
        long long above = 0;
        for (int r2 = 0; r2 < R; ++r2)
            if (a.run_key[r2] > key) above += (a.run_start[r2 + 1] - a.run_start[r2]) - a.run_take[r2];
        const long long f = min(left, max(0LL, fill - above));
        a.mask[a.len + r] = (int)(a.run_take[r] + f);  // staged per-run keep count
    }
    __syncthreads();

    // ---- keep mask over slots: sinks, window, newest kept tokens of each run
    for (int i = tid; i < a.len; i += SEL_THREADS) a.mask[i] = (i < a.n_s || i >= c1) ? 1 : 0;
    __syncthreads();
    for (int r = tid; r < R; r += SEL_THREADS) {
        const int e = a.run_start[r + 1], kcount = a.mask[a.len + r];
        for (int i = e - kcount; i < e; ++i) a.mask[i] = 1;
    }
    __syncthreads();

    // ---- keep list (ascending) and its inverse on destinations [0, M)
    {
        const int per = (a.len + SEL_THREADS - 1) / SEL_THREADS;
        const int lo = tid * per, hi = min(lo + per, a.len);
        int cnt = 0;
        for (int i = lo; i < hi; ++i) cnt += a.mask[i];
        int tot = 0;
        int off = block_excl_scan(cnt, s_scan, tot);
        for (int i = lo; i < hi; ++i) {
            if (a.mask[i]) {
                if (off < a.M) {
                    a.keep[off] = i;
                    if (a.keep_out) a.keep_out[off] = i;
                }
                if (i < a.M) a.inv[i] = off;
                ++off;
            } else if (i < a.M) {
                a.inv[i] = -1;
            }
        }
        if (tid == 0 && tot != a.M) {  // cannot happen for valid arguments; never move data then
            a.status[0] = 2;
            a.status[1] = 1;
        }
    }
}

struct GatherArgs {
    char *planes[KV_MAX_PLANES];
    int n_planes, row_bytes, M, n_chunks;
    long long total_bytes;  // n_planes * row_bytes
    int32_t *pos, *chunk;
    const int32_t *keep, *inv;
    int32_t *flags, *status;
    uint32_t *ticket;
};

__global__ __launch_bounds__(256) void kv_gather_kernel(GatherArgs a) {
    __shared__ int s_t;
    if (a.status[1]) return;
    const int tid = threadIdx.x;
    if (tid == 0) s_t = (int)atomicAdd(a.ticket, 1u);
    __syncthreads();
    const int t = s_t;
    const int d = t / a.n_chunks, c = t % a.n_chunks;
    if (d >= a.M) return;
    const int src = a.keep[d];
    if (src == d) return;  // row already in place; nobody else reads it

    // ---- read the source row (this group's 64 KiB piece of it)
    uint4 buf[GATHER_U];
    const long long base = (long long)c * GATHER_BYTES;
#pragma unroll
    for (int u = 0; u < GATHER_U; ++u) {
        const long long o = base + 16LL * (tid + 256 * u);
        if (o < a.total_bytes) {
            const int p = (int)(o / a.row_bytes), wi = (int)(o % a.row_bytes);
            buf[u] = *(const uint4 *)(a.planes[p] + (size_t)src * a.row_bytes + wi);
        }
    }
    int pv = 0, cv = 0;
    if (c == 0 && tid == 0) {
        pv = a.pos[src];
        cv = a.chunk[src];
    }
    __builtin_amdgcn_s_waitcnt(0);  // every load of this thread has returned
    __syncthreads();
    if (tid == 0) __hip_atomic_store(&a.flags[t], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);

    // ---- wait until the reader of row d (a lower ticket) holds its data
    if (tid == 0) {
        const int dep = a.inv[d];
        if (dep >= 0 && dep != d) {
            int it = 0;
            const int ft = dep * a.n_chunks + c;
            while (__hip_atomic_load(&a.flags[ft], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
                if (++it >= SPIN_LIMIT) {
                    __hip_atomic_store(&a.status[2], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    break;
                }
                __builtin_amdgcn_s_sleep(2);
            }
        }
    }
    __syncthreads();

    // ---- write slot d
#pragma unroll
    for (int u = 0; u < GATHER_U; ++u) {
        const long long o = base + 16LL * (tid + 256 * u);
        if (o < a.total_bytes) {
            const int p = (int)(o / a.row_bytes), wi = (int)(o % a.row_bytes);
            *(uint4 *)(a.planes[p] + (size_t)d * a.row_bytes + wi) = buf[u];
        }
    }
    if (c == 0 && tid == 0) {
        a.pos[d] = pv;
        a.chunk[d] = cv;
    }
}

static size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

KvWorkspace kv_workspace_layout(int n_layers, int row_bytes, int capacity) {
    KvWorkspace w{};
    const long long total = 2LL * n_layers * row_bytes;
    w.n_chunks = (int)((total + GATHER_BYTES - 1) / GATHER_BYTES);
    if (w.n_chunks < 1) w.n_chunks = 1;
    const size_t cap = (size_t)capacity;
    size_t off = 0;
    w.offStatus = off;
    off = align256(off + 64);
    w.offKeep = off;
    off = align256(off + cap * 4);
    w.offInv = off;
    off = align256(off + cap * 4);
    w.offMask = off;
    off = align256(off + 2 * cap * 4);  // slot mask + per-run keep counts
    w.offRunStart = off;
    off = align256(off + (cap + 1) * 4);
    w.offRunKey = off;
    off = align256(off + cap * 8);
    w.offRunBkt = off;
    off = align256(off + cap * 4);
    w.offRunTake = off;
    off = align256(off + cap * 4);
    w.offFlags = off;
    off = align256(off + cap * (size_t)w.n_chunks * 4);
    w.total = off;
    return w;
}

hipError_t launch_kv_evict(const KvLaunch &p, hipStream_t stream) {
    char *ws = p.ws;
    KvArgs a;
    a.pos_in = p.pos;
    a.chunk = p.chunk_id;
    a.scores = p.chunk_scores;
    a.num_chunks = p.num_chunks;
    a.len = p.len;
    a.M = p.M;
    a.n_s = p.n_sink;
    a.n_w = p.n_window;
    a.N = p.n_buckets;
    a.n_flags = p.M * p.lay.n_chunks;
    a.status = (int32_t *)(ws + p.lay.offStatus);
    a.ticket = (uint32_t *)(ws + p.lay.offStatus + 32);
    a.keep = (int32_t *)(ws + p.lay.offKeep);
    a.inv = (int32_t *)(ws + p.lay.offInv);
    a.mask = (int32_t *)(ws + p.lay.offMask);
    a.run_start = (int32_t *)(ws + p.lay.offRunStart);
    a.run_key = (unsigned long long *)(ws + p.lay.offRunKey);
    a.run_bkt = (int32_t *)(ws + p.lay.offRunBkt);
    a.run_take = (int32_t *)(ws + p.lay.offRunTake);
    a.flags = (int32_t *)(ws + p.lay.offFlags);
    a.keep_out = p.keep_out;
    hipLaunchKernelGGL(kv_select_kernel, dim3(1), dim3(SEL_THREADS), 0, stream, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

    GatherArgs g;
    for (int i = 0; i < KV_MAX_PLANES; ++i) g.planes[i] = i < p.n_planes ? p.planes[i] : nullptr;
    g.n_planes = p.n_planes;
    g.row_bytes = p.row_bytes;
    g.M = p.M;
    g.n_chunks = p.lay.n_chunks;
    g.total_bytes = (long long)p.n_planes * p.row_bytes;
    g.pos = p.pos;
    g.chunk = p.chunk_id;
    g.keep = a.keep;
    g.inv = a.inv;
    g.flags = a.flags;
    g.status = a.status;
    g.ticket = a.ticket;
    const long long groups = (long long)p.M * p.lay.n_chunks;
    if (groups == 0) return hipSuccess;
    hipLaunchKernelGGL(kv_gather_kernel, dim3((unsigned)groups), dim3(256), 0, stream, g);
    return hipGetLastError();
}

}  // namespace ds
