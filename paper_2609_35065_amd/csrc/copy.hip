// copy.hip -- retrieve scatter and store gather between staged chunks and
// paged KV blocks, for CDNA4 (gfx950).
//
// Vocabulary.  A segment is the B tokens of one layer's K or V plane that
// form one paged block: B*H*D*e contiguous bytes on both sides (32 KiB for
// block 16 x 8 heads x 128 dims x bf16).  A unit is the C/B segments of one
// (job, layer, plane): contiguous in the staged chunk, one paged block each.
// A row is one 16-byte vector per lane of a workgroup (T*16 bytes, one wave
// instruction per 64 lanes covering 1 KiB of contiguous memory).
//
// Retrieve (staging -> paged), fast path: one 256-lane workgroup per unit.
// The unit's staged bytes are read front to back in stages of 8 vectors per
// lane; the loads of stage s+1 are issued before the stores of stage s, and
// the workgroup waits for both before going on, so it keeps one segment of
// writes in flight (more was measured slower where chunks are shared).
// Block ids come through the scalar cache.
// Units are ordered (layer, plane)-major and job-minor, and each of the 8
// XCDs walks one contiguous range of that order, so the jobs that share a
// staged chunk (requests reusing one prefix; adjacent once the job list is
// grouped by slot) read the same 512 KiB back to back through one XCD's L2.
// Loads are cached; paged writes are non-temporal.
//
// Store (paged -> staging), fast path: 1024-lane workgroups, each copying a
// group of segments with 16 vectors per lane in flight (256 KiB per
// workgroup for 32 KiB segments), all loads before all stores; job-major
// order, each XCD taking one contiguous range of it, so a die fills whole
// staging slots front to back.  Both loads and stores are non-temporal: each
// byte is touched once.  The same kernel in the other direction is the
// streaming retrieve, for job lists in which no staged chunk is read twice:
// there is no reuse to keep in cache, and it is 3-6 % faster than the unit
// walk on such lists (much slower where chunks are shared).
//
// The pair retrieve walks two consecutive jobs per workgroup and, when they
// name one staged chunk, loads each stage once for both: with groups of 8
// requests per chunk it is 3-13 % faster than the unit walk.  The host picks
// among these three retrieves from the job list (kv_retrieve_plan).  A fourth,
// the four-job-window retrieve (one segment of four consecutive jobs per
// 1024-lane workgroup), is faster than the pair walk on pools where the memory
// system takes scattered writes slowly and slower elsewhere, so the caller
// picks it by timing.
//
// On MI355X these shapes were chosen by measurement: at 256 lanes a plain
// contiguous copy tops out near 5.2 TB/s (read + write), at 1024 lanes near
// 5.9 TB/s; the 256-lane walks are the fastest retrieves where chunks are
// shared because their stores are scattered 32 KiB blocks while their loads
// hit in cache.
//
// Generic path: any segment size that is a multiple of 16 bytes, one
// 256-lane workgroup per segment.

#include "internal.h"

namespace tkv {
namespace {

typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef int32_t v4i __attribute__((ext_vector_type(4)));
// Uniform reads through the scalar cache: loads from the constant address
// space with wave-uniform addresses become s_load instructions.
typedef const __attribute__((address_space(4))) v4i *const_job_ptr;
typedef const __attribute__((address_space(4))) int32_t *const_i32_ptr;

template <bool kNT>
__device__ __forceinline__ v4u load16(const v4u *p) {
    if constexpr (kNT) return __builtin_nontemporal_load(p);
    else return *p;
}

__device__ __forceinline__ bool job_ok(const CopyParams &p, const v4i jb) {
    return jb.x >= 0 && jb.x < p.num_slots && jb.y >= 0 && jb.y < p.num_reqs && jb.z >= 0 &&
           ((int64_t)jb.z + 1) * p.nseg <= p.bt_stride;
}

__device__ __forceinline__ bool blk_ok(const CopyParams &p, int32_t blk) {
    return blk >= 0 && blk < p.num_blocks;
}

// Accelerator complex dies on MI355X; consecutive workgroups of a launch are
// dispatched to them round-robin.  Only performance depends on this value.
constexpr int kXcds = 8;

// --------------------------------------------------------------------------
// Retrieve fast path: R rows of 4 KiB per segment (segment = R * 4 KiB).
// --------------------------------------------------------------------------
template <int R>
__global__ __launch_bounds__(256) void retrieve_unit_kernel(CopyParams p) {
    constexpr int T = 256;
    constexpr int SB = R >= 8 ? 1 : 8 / R;   // segments per pipeline stage
    constexpr int V = R * SB;                // vectors per lane per stage
    const int tid = threadIdx.x;
    const int64_t units = (int64_t)p.num_jobs * p.L * 2;
    const int64_t per_xcd = (units + kXcds - 1) / kXcds;
    const int32_t nstage = (p.nseg + SB - 1) / SB;
    // XCD-aware order: workgroup b runs on XCD b mod 8, so XCD x walks the
    // contiguous range [x*per_xcd, (x+1)*per_xcd) of the unit order; the
    // grid (and its stride) is a multiple of kXcds.
    for (int64_t w = blockIdx.x; w < per_xcd * kXcds; w += gridDim.x) {
        const int64_t u = (w % kXcds) * per_xcd + w / kXcds;
        if (u >= units) continue;
        const int64_t q = u % p.num_jobs;
        const int64_t t = u / p.num_jobs;
        const int32_t kv = (int32_t)(t & 1);
        const int32_t l = (int32_t)(t >> 1);
        const v4i jb = ((const_job_ptr)p.jobs)[q];
        if (!job_ok(p, jb)) continue;
        const const_i32_ptr btp = (const_i32_ptr)p.bt + (int64_t)jb.y * p.bt_stride + (int64_t)jb.z * p.nseg;
        const v4u *src = reinterpret_cast<const v4u *>(p.staging + (int64_t)jb.x * p.slot_bytes +
                                                       ((int64_t)l * 2 + kv) * p.nseg * p.seg_bytes) + tid;
        char *dst_plane = p.layers[l] + kv * p.kv_stride;

        v4u a[V], b[V];
#pragma unroll
        for (int k = 0; k < V; ++k)
            if (k / R < p.nseg) a[k] = src[(int64_t)k * T];
        for (int32_t s = 0; s < nstage; ++s) {
            const int32_t s0 = s * SB;
            if (s + 1 < nstage) {
                const v4u *nsrc = src + (int64_t)(s0 + SB) * R * T;
#pragma unroll
                for (int k = 0; k < V; ++k)
                    if (s0 + SB + k / R < p.nseg) b[k] = nsrc[(int64_t)k * T];
            }
#pragma unroll
            for (int j = 0; j < SB; ++j) {
                const int32_t seg = s0 + j;
                if (seg >= p.nseg) break;
                const int32_t blk = btp[seg];
                if (!blk_ok(p, blk)) continue;
                v4u *dst = reinterpret_cast<v4u *>(dst_plane + (int64_t)blk * p.block_stride) + tid;
#pragma unroll
                for (int r = 0; r < R; ++r) __builtin_nontemporal_store(a[j * R + r], dst + r * T);
            }
#pragma unroll
            for (int k = 0; k < V; ++k) a[k] = b[k];
        }
    }
}

// --------------------------------------------------------------------------
// Retrieve, pairs of jobs (32 KiB segments): a unit is (jobs 2w and 2w+1,
// layer, plane).  When both jobs name the same staged chunk, each stage of it
// is loaded once and stored to both jobs' blocks; otherwise each job is walked
// on its own.  Stages are ping-ponged between two register sets, and the
// loads of the last stage are clamped to the unit so that every stage issues
// the same instructions.
// --------------------------------------------------------------------------
template <int R, bool kTwo>
__device__ __forceinline__ void pair_walk(const CopyParams &p, const char *src, const_i32_ptr rows0,
                                          const_i32_ptr rows1, char *dst_plane, int tid) {
    constexpr int T = 256;
    constexpr int V = R;
    const int32_t ns = p.nseg;
    const int64_t seg = p.seg_bytes;
    const v4u *base = reinterpret_cast<const v4u *>(src) + tid;
    v4u A[V], B[V];
#pragma unroll
    for (int x = 0; x < V; ++x) A[x] = base[x * T];
    for (int32_t s = 0; s < ns; s += 2) {
        const int32_t s1 = s + 1 < ns ? s + 1 : ns - 1;
        const v4u *n1 = reinterpret_cast<const v4u *>(src + (int64_t)s1 * seg) + tid;
#pragma unroll
        for (int x = 0; x < V; ++x) B[x] = n1[x * T];
        {
            const int32_t b0 = rows0[s];
            if (blk_ok(p, b0)) {
                v4u *d = reinterpret_cast<v4u *>(dst_plane + (int64_t)b0 * p.block_stride) + tid;
#pragma unroll
                for (int x = 0; x < V; ++x) __builtin_nontemporal_store(A[x], d + x * T);
            }
            if constexpr (kTwo) {
                const int32_t b1 = rows1[s];
                if (blk_ok(p, b1)) {
                    v4u *d = reinterpret_cast<v4u *>(dst_plane + (int64_t)b1 * p.block_stride) + tid;
#pragma unroll
                    for (int x = 0; x < V; ++x) __builtin_nontemporal_store(A[x], d + x * T);
                }
            }
        }
        if (s + 1 >= ns) break;
        const int32_t s2 = s + 2 < ns ? s + 2 : ns - 1;
        const v4u *n2 = reinterpret_cast<const v4u *>(src + (int64_t)s2 * seg) + tid;
#pragma unroll
        for (int x = 0; x < V; ++x) A[x] = n2[x * T];
        {
            const int32_t b0 = rows0[s + 1];
            if (blk_ok(p, b0)) {
                v4u *d = reinterpret_cast<v4u *>(dst_plane + (int64_t)b0 * p.block_stride) + tid;
#pragma unroll
                for (int x = 0; x < V; ++x) __builtin_nontemporal_store(B[x], d + x * T);
            }
            if constexpr (kTwo) {
                const int32_t b1 = rows1[s + 1];
                if (blk_ok(p, b1)) {
                    v4u *d = reinterpret_cast<v4u *>(dst_plane + (int64_t)b1 * p.block_stride) + tid;
#pragma unroll
                    for (int x = 0; x < V; ++x) __builtin_nontemporal_store(B[x], d + x * T);
                }
            }
        }
    }
}

template <int R>
__global__ __launch_bounds__(256) void retrieve_pair_kernel(CopyParams p) {
    const int tid = threadIdx.x;
    const int64_t npair = ((int64_t)p.num_jobs + 1) / 2;
    const int64_t units = npair * p.L * 2;
    const int64_t per_xcd = (units + kXcds - 1) / kXcds;
    const const_job_ptr jobs = (const_job_ptr)p.jobs;
    // the unit order and XCD ranges of retrieve_unit_kernel, over pairs
    for (int64_t w = blockIdx.x; w < per_xcd * kXcds; w += gridDim.x) {
        const int64_t u = (w % kXcds) * per_xcd + w / kXcds;
        if (u >= units) continue;
        const int64_t q0 = 2 * (u % npair);
        const int64_t t = u / npair;
        const int32_t kv = (int32_t)(t & 1);
        const int32_t l = (int32_t)(t >> 1);
        const bool has1 = q0 + 1 < p.num_jobs;
        const v4i j0 = jobs[q0];
        const v4i j1 = has1 ? jobs[q0 + 1] : v4i{-1, -1, -1, 0};
        const bool ok0 = job_ok(p, j0);
        const bool ok1 = has1 && job_ok(p, j1);
        char *dst_plane = p.layers[l] + kv * p.kv_stride;
        const int64_t plane_off = ((int64_t)l * 2 + kv) * p.nseg * p.seg_bytes;
        const const_i32_ptr rows0 = (const_i32_ptr)p.bt + (ok0 ? (int64_t)j0.y * p.bt_stride + (int64_t)j0.z * p.nseg : 0);
        const const_i32_ptr rows1 = (const_i32_ptr)p.bt + (ok1 ? (int64_t)j1.y * p.bt_stride + (int64_t)j1.z * p.nseg : 0);
        if (ok0 && ok1 && j0.x == j1.x) {
            pair_walk<R, true>(p, p.staging + (int64_t)j0.x * p.slot_bytes + plane_off, rows0, rows1, dst_plane, tid);
        } else {
            if (ok0) pair_walk<R, false>(p, p.staging + (int64_t)j0.x * p.slot_bytes + plane_off, rows0, rows0, dst_plane, tid);
            if (ok1) pair_walk<R, false>(p, p.staging + (int64_t)j1.x * p.slot_bytes + plane_off, rows1, rows1, dst_plane, tid);
        }
    }
}

// --------------------------------------------------------------------------
// Retrieve, windows of four jobs (R rows of 4 KiB per segment): a unit is
// (layer, plane, window of jobs 4w..4w+3, segment s), copied by one 1024-lane
// workgroup whose quarter j moves job 4w+j's segment s.  Jobs of a window that
// share a staged chunk load the same bytes at the same time, so one load comes
// from memory and the others from L2.  Units are (layer, plane)-major, then
// groups of kQuadGroup windows (32 jobs), then segment, then window, in plain
// dispatch order: the workgroups in flight write one segment of 32 jobs at a
// time.  (Window-major order, and groups of 1, 2 or 4 windows, measured 2-7 %
// slower.)
// --------------------------------------------------------------------------
constexpr int kQuadGroup = 8;

template <int R>
__global__ __launch_bounds__(1024) void retrieve_quad_kernel(CopyParams p) {
    constexpr int T = 256;
    // the quarter is uniform within each 64-lane wave
    const int j = __builtin_amdgcn_readfirstlane(threadIdx.x >> 8);
    const int tid = threadIdx.x & (T - 1);
    const int64_t ngroup = ((int64_t)p.num_jobs + 4 * kQuadGroup - 1) / (4 * kQuadGroup);
    const int64_t units = ngroup * kQuadGroup * p.nseg * p.L * 2;
    for (int64_t u = blockIdx.x; u < units; u += gridDim.x) {
        const int32_t h = (int32_t)(u % kQuadGroup);
        const int64_t t = u / kQuadGroup;
        const int32_t s = (int32_t)(t % p.nseg);
        const int64_t g = t / p.nseg;
        const int64_t q = ((g % ngroup) * kQuadGroup + h) * 4 + j;
        const int64_t pl = g / ngroup;   // layer * 2 + plane
        if (q >= p.num_jobs) continue;
        const v4i jb = ((const_job_ptr)p.jobs)[q];
        if (!job_ok(p, jb)) continue;
        const int32_t blk = ((const_i32_ptr)p.bt)[(int64_t)jb.y * p.bt_stride + (int64_t)jb.z * p.nseg + s];
        if (!blk_ok(p, blk)) continue;
        const int32_t kv = (int32_t)(pl & 1);
        const int32_t l = (int32_t)(pl >> 1);
        const v4u *src = reinterpret_cast<const v4u *>(p.staging + (int64_t)jb.x * p.slot_bytes +
                                                       (pl * p.nseg + s) * p.seg_bytes) + tid;
        v4u *dst = reinterpret_cast<v4u *>(p.layers[l] + kv * p.kv_stride + (int64_t)blk * p.block_stride) + tid;
        v4u a[R];
#pragma unroll
        for (int r = 0; r < R; ++r) a[r] = src[r * T];
#pragma unroll
        for (int r = 0; r < R; ++r) __builtin_nontemporal_store(a[r], dst + r * T);
    }
}

// --------------------------------------------------------------------------
// Group fast path (store, streaming retrieve): T lanes, R rows of T*16 bytes
// per segment, SPW segments per workgroup (R * SPW = 16 vectors per lane).
// --------------------------------------------------------------------------
template <int T, int R, bool kRetrieve>
__global__ __launch_bounds__(T) void group_copy_kernel(CopyParams p) {
    constexpr int SPW = 16 / R;
    constexpr int V = R * SPW;
    const int tid = threadIdx.x;
    const int32_t gpu = (p.nseg + SPW - 1) / SPW;
    const int64_t total = (int64_t)p.num_jobs * p.L * 2 * gpu;
    const int64_t per_xcd = (total + kXcds - 1) / kXcds;
    // XCD x copies the contiguous range [x*per_xcd, (x+1)*per_xcd) of the
    // job-major group order: whole staging slots per die.
    for (int64_t w = blockIdx.x; w < per_xcd * kXcds; w += gridDim.x) {
        const int64_t g = (w % kXcds) * per_xcd + w / kXcds;
        if (g >= total) continue;
        const int32_t ig = (int32_t)(g % gpu);
        int64_t t = g / gpu;
        const int32_t kv = (int32_t)(t & 1);
        t >>= 1;
        const int32_t l = (int32_t)(t % p.L);
        const int64_t q = t / p.L;
        const v4i jb = ((const_job_ptr)p.jobs)[q];
        if (!job_ok(p, jb)) continue;
        const int32_t s0 = ig * SPW;
        const const_i32_ptr btp = (const_i32_ptr)p.bt + (int64_t)jb.y * p.bt_stride + (int64_t)jb.z * p.nseg + s0;
        int32_t blk[SPW];
#pragma unroll
        for (int j = 0; j < SPW; ++j) blk[j] = (s0 + j < p.nseg) ? btp[j] : -1;
        char *plane = p.layers[l] + kv * p.kv_stride;
        v4u *stg = reinterpret_cast<v4u *>(p.staging + (int64_t)jb.x * p.slot_bytes +
                                           (((int64_t)l * 2 + kv) * p.nseg + s0) * p.seg_bytes) + tid;
        v4u r[V];
        if constexpr (kRetrieve) {
            // staged segments s0.. are contiguous; a segment whose block id is invalid is read but not written
#pragma unroll
            for (int k = 0; k < V; ++k)
                if (s0 + k / R < p.nseg) r[k] = __builtin_nontemporal_load(stg + (int64_t)k * T);
#pragma unroll
            for (int k = 0; k < V; ++k) {
                const int j = k / R;
                if (blk_ok(p, blk[j])) {
                    v4u *dst = reinterpret_cast<v4u *>(plane + (int64_t)blk[j] * p.block_stride) + tid;
                    __builtin_nontemporal_store(r[k], dst + (k % R) * T);
                }
            }
        } else {
#pragma unroll
            for (int k = 0; k < V; ++k) {
                const int j = k / R;
                if (blk_ok(p, blk[j])) {
                    const v4u *src = reinterpret_cast<const v4u *>(plane + (int64_t)blk[j] * p.block_stride) + tid;
                    r[k] = __builtin_nontemporal_load(src + (k % R) * T);
                }
            }
#pragma unroll
            for (int k = 0; k < V; ++k)
                if (blk_ok(p, blk[k / R])) __builtin_nontemporal_store(r[k], stg + (int64_t)k * T);
        }
    }
}

// --------------------------------------------------------------------------
// Generic path: one 256-lane workgroup per segment, any multiple of 16 bytes.
// --------------------------------------------------------------------------
constexpr int kGenThreads = 256;
constexpr int kGenUnroll = 8;

template <bool kSrcNT>
__device__ __forceinline__ void copy_segment(v4u *__restrict__ dst, const v4u *__restrict__ src, int64_t bytes,
                                             int tid) {
    const int64_t n = bytes >> 4;
    for (int64_t base = 0; base < n; base += (int64_t)kGenThreads * kGenUnroll) {
        v4u r[kGenUnroll];
#pragma unroll
        for (int k = 0; k < kGenUnroll; ++k) {
            const int64_t v = base + k * kGenThreads + tid;
            if (v < n) r[k] = load16<kSrcNT>(src + v);
        }
#pragma unroll
        for (int k = 0; k < kGenUnroll; ++k) {
            const int64_t v = base + k * kGenThreads + tid;
            if (v < n) __builtin_nontemporal_store(r[k], dst + v);
        }
    }
}

template <bool kRetrieve>
__global__ __launch_bounds__(kGenThreads) void copy_generic_kernel(CopyParams p) {
    const int tid = threadIdx.x;
    const int64_t total = (int64_t)p.num_jobs * p.L * 2 * p.nseg;
    for (int64_t g = blockIdx.x; g < total; g += gridDim.x) {
        const int64_t q = g % p.num_jobs;
        int64_t t = g / p.num_jobs;
        const int32_t i = (int32_t)(t % p.nseg);
        t /= p.nseg;
        const int32_t kv = (int32_t)(t & 1);
        const int32_t l = (int32_t)(t >> 1);
        const v4i jb = ((const_job_ptr)p.jobs)[q];
        if (!job_ok(p, jb)) continue;
        const int32_t blk = ((const_i32_ptr)p.bt)[(int64_t)jb.y * p.bt_stride + (int64_t)jb.z * p.nseg + i];
        if (!blk_ok(p, blk)) continue;
        char *stg = p.staging + (int64_t)jb.x * p.slot_bytes + (((int64_t)l * 2 + kv) * p.nseg + i) * p.seg_bytes;
        char *pg = p.layers[l] + kv * p.kv_stride + (int64_t)blk * p.block_stride;
        if constexpr (kRetrieve)
            copy_segment<false>(reinterpret_cast<v4u *>(pg), reinterpret_cast<const v4u *>(stg), p.seg_bytes, tid);
        else
            copy_segment<true>(reinterpret_cast<v4u *>(stg), reinterpret_cast<const v4u *>(pg), p.seg_bytes, tid);
    }
}

constexpr int64_t kMaxGrid = int64_t(1) << 30;

unsigned grid_of(int64_t items) { return (unsigned)(items < kMaxGrid ? items : kMaxGrid); }

template <int R>
void launch_retrieve_unit(const CopyParams &p, hipStream_t s) {
    const int64_t units = (int64_t)p.num_jobs * p.L * 2;
    const int64_t grid = (units + kXcds - 1) / kXcds * kXcds;   // kMaxGrid is a multiple of kXcds too
    hipLaunchKernelGGL(retrieve_unit_kernel<R>, dim3(grid_of(grid)), dim3(256), 0, s, p);
}

template <int T, int R, bool kRetrieve>
void launch_group(const CopyParams &p, hipStream_t s) {
    const int64_t gpu = (p.nseg + 16 / R - 1) / (16 / R);
    const int64_t total = (int64_t)p.num_jobs * p.L * 2 * gpu;
    hipLaunchKernelGGL((group_copy_kernel<T, R, kRetrieve>), dim3(grid_of((total + kXcds - 1) / kXcds * kXcds)),
                       dim3(T), 0, s, p);
}

// Rows of `row_bytes` per segment if the segment is 1, 2, 4, 8 or 16 rows.
int rows_of(int64_t seg_bytes, int64_t row_bytes) {
    if (seg_bytes % row_bytes) return 0;
    const int64_t r = seg_bytes / row_bytes;
    return (r == 1 || r == 2 || r == 4 || r == 8 || r == 16) ? (int)r : 0;
}

bool launch_retrieve_pair(const CopyParams &p, hipStream_t s) {
    if (rows_of(p.seg_bytes, 256 * 16) != 8) return false;   // measured at 32 KiB segments only
    const int64_t units = ((int64_t)p.num_jobs + 1) / 2 * p.L * 2;
    const int64_t grid = (units + kXcds - 1) / kXcds * kXcds;
    hipLaunchKernelGGL(retrieve_pair_kernel<8>, dim3(grid_of(grid)), dim3(256), 0, s, p);
    return true;
}

template <int R>
void launch_retrieve_quad_r(const CopyParams &p, hipStream_t s) {
    const int64_t units = ((int64_t)p.num_jobs + 4 * kQuadGroup - 1) / (4 * kQuadGroup) * kQuadGroup * p.nseg * p.L * 2;
    hipLaunchKernelGGL(retrieve_quad_kernel<R>, dim3(grid_of(units)), dim3(1024), 0, s, p);
}

bool launch_retrieve_quad(const CopyParams &p, hipStream_t s) {
    switch (rows_of(p.seg_bytes, 256 * 16)) {
    case 1: launch_retrieve_quad_r<1>(p, s); return true;
    case 2: launch_retrieve_quad_r<2>(p, s); return true;
    case 4: launch_retrieve_quad_r<4>(p, s); return true;
    case 8: launch_retrieve_quad_r<8>(p, s); return true;
    case 16: launch_retrieve_quad_r<16>(p, s); return true;
    default: return false;
    }
}

bool launch_retrieve_fast(const CopyParams &p, hipStream_t s) {
    switch (rows_of(p.seg_bytes, 256 * 16)) {
    case 1: launch_retrieve_unit<1>(p, s); return true;
    case 2: launch_retrieve_unit<2>(p, s); return true;
    case 4: launch_retrieve_unit<4>(p, s); return true;
    case 8: launch_retrieve_unit<8>(p, s); return true;
    case 16: launch_retrieve_unit<16>(p, s); return true;
    default: return false;
    }
}

template <int T, bool kRetrieve>
bool launch_group_t(const CopyParams &p, hipStream_t s) {
    switch (rows_of(p.seg_bytes, (int64_t)T * 16)) {
    case 1: launch_group<T, 1, kRetrieve>(p, s); return true;
    case 2: launch_group<T, 2, kRetrieve>(p, s); return true;
    case 4: launch_group<T, 4, kRetrieve>(p, s); return true;
    case 8: launch_group<T, 8, kRetrieve>(p, s); return true;
    case 16: launch_group<T, 16, kRetrieve>(p, s); return true;
    default: return false;
    }
}

template <bool kRetrieve>
bool launch_group_fast(const CopyParams &p, hipStream_t s) {
    return launch_group_t<1024, kRetrieve>(p, s) || launch_group_t<512, kRetrieve>(p, s) ||
           launch_group_t<256, kRetrieve>(p, s);
}

}  // namespace

hipError_t launch_copy(const CopyParams &p, CopyKind kind, hipStream_t stream) {
    if (p.total_segs <= 0) return hipSuccess;
    (void)hipGetLastError();   // clear an error left by an unrelated earlier call
    const bool retrieve = kind != kStore;
    const bool fast = kind == kRetrieve         ? launch_retrieve_fast(p, stream)
                      : kind == kRetrievePair   ? launch_retrieve_pair(p, stream) || launch_retrieve_fast(p, stream)
                      : kind == kRetrieveQuad   ? launch_retrieve_quad(p, stream)
                      : kind == kRetrieveStream ? launch_group_fast<true>(p, stream)
                                                : launch_group_fast<false>(p, stream);
    if (!fast) {
        const unsigned grid = grid_of(p.total_segs);
        if (retrieve)
            hipLaunchKernelGGL(copy_generic_kernel<true>, dim3(grid), dim3(kGenThreads), 0, stream, p);
        else
            hipLaunchKernelGGL(copy_generic_kernel<false>, dim3(grid), dim3(kGenThreads), 0, stream, p);
    }
    return hipGetLastError();
}

}  // namespace tkv
