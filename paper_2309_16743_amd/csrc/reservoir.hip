// GPU-resident training buffers of Sec. 3.2.3: the paper's Algorithm 1
// ("Reservoir") as slot-encoded device state plus four kernels per operation
// pair (put: assign + copy, sample: select + gather), and the two comparison
// buffers that evict a sample when it is read, FIFO and FIRO, over the same
// slabs, gather and copy kernels.
//
// FIFO / FIRO state: the list of stored samples `occ` is a ring of C
// positions starting at occ_base; free slots form a second ring `free_q`
// (head free_head, C - N entries): a put takes slots from its head and
// appends them to the list, a batch takes samples out of the list (FIFO: the
// first B; FIRO: B positions by partial Fisher-Yates) and pushes their slots
// at the free queue's tail.  All ring positions are known on the host.
//
// State on the device: an x slab (C x ldxs fp32) and a u slab (C x ldus fp32),
// per-slot seen counts (int32, -1 = empty slot) and sample ids (int64), the
// drain order `occ` (int32, used after reception ends), a histogram of seen
// counts of samples that left the buffer, and a counter block.  In the normal
// phase (reception not over) the occupied slots are exactly [0, N), so the
// draw index is the slot.
//
// Every state-changing call runs in ticket order on the reservoir's ordering
// stream, so the device state after ticket p depends only on the calls with
// tickets <= p.  N is known on the host from the call sequence alone: a put
// of k rows leaves N = min(C, N + k) (each row fills a free slot or replaces a
// seen sample, and a = min(k, C - U) >= min(k, C - N)); a drain batch removes
// min(b, N).  So readiness (N > T) never needs a device read-back.
#include <algorithm>
#include <mutex>
#include <vector>

#include "common.h"
#include "philox.h"
#include "res_host.h"
#include "reservoir.h"

namespace ot {

constexpr int kHistLen = 64;           // eviction histogram buckets (last = overflow)
constexpr int kTile = 1024;            // slots per tile of the seen-count index
constexpr int64_t kMaxPut = 4096;      // rows per put (bounded LDS of the assign kernel)
constexpr int64_t kMaxDrainBatch = 4096;
constexpr int64_t kMaxBatch = 65536;
constexpr int kAssignThreads = 1024;

struct ResCounters {
  long long U, S, N, total_put, total_evicted, total_deleted, total_draws, next_sample_id;
  long long last_accepted;   // a of the last put
  long long last_free;       // F of the last put
  long long last_evicted;    // E of the last put
  long long last_base_id;    // first sample id of the last put
  long long pad[4];
};

// ------------------------------------------------------------------ device helpers
__device__ inline void atomic_add_ll(long long* p, long long v) {
  atomicAdd(reinterpret_cast<unsigned long long*>(p), static_cast<unsigned long long>(v));
}

// Exclusive scan of one int per thread over a block of NT threads.
template <int NT>
__device__ int block_exclusive_scan(int v, int* wave_tot, int* total) {
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    int t = __shfl_up(incl, off, 64);
    if (lane >= off) incl += t;
  }
  if (lane == 63) wave_tot[wid] = incl;
  __syncthreads();
  if (wid == 0) {
    const int w = lane < NT / 64 ? wave_tot[lane] : 0;
    int wi = w;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      int t = __shfl_up(wi, off, 64);
      if (lane >= off) wi += t;
    }
    if (lane < NT / 64) wave_tot[lane] = wi - w;
    if (lane == NT / 64 - 1) *total = wi;
  }
  __syncthreads();
  return incl - v + wave_tot[wid];
}

// Partial Fisher-Yates over a virtual array A (A[p] = base[p]) without
// materialising the swaps.  Step j (0 <= j < E) swaps A[j] and A[r_j]
// (r_j >= j) and takes A[j].  Position j is never touched after step j, so:
//   pre_j   = A[j] just before step j = pre_i for the latest i < j with r_i = j,
//             else base[j];
//   taken_j = A[r_j] just before step j = pre_j if r_j = j, else pre_i for the
//             latest i < j with r_i = r_j, else base[r_j].
// The latest-writer queries go through a hash table of the steps keyed by
// r_i (open addressing in LDS, at most half full, so every probe sequence
// ends at an empty entry; the draws rarely collide, so most queries read one
// or two entries), and the pre_j chains are resolved by pointer jumping,
// skipped when no step has a predecessor.  Inputs: r[0..E) in LDS, a table of
// 2^tbits ints (2^tbits >= 2 E).  Outputs: pre[0..E), taken[0..E) in LDS;
// last_writer[j] = 1 when no later step writes position r_j (used by the
// drain to persist the shuffle).  base(p) returns base[p] (the identity for
// the eviction list).
constexpr int kShuffleArrays = 7;       // r, par, par2, lv, pre, taken, last_writer
__host__ __device__ inline int shuffle_table_bits(int64_t cap) {
  int b = 1;
  while ((int64_t(1) << b) < 2 * cap) ++b;
  return b;
}
// ints of dynamic LDS that a kernel resolving a shuffle of up to cap steps
// needs: the seven arrays and the hash table
__host__ __device__ inline int64_t shuffle_lds_ints(int64_t cap) {
  return kShuffleArrays * cap + (int64_t(1) << shuffle_table_bits(cap));
}

template <class Base>
__device__ void resolve_partial_shuffle(int E, const int* r, Base base, int* table, int tbits, int* par, int* par2,
                                        int* lv, int* pre, int* taken, int* last_writer) {
  const int nt = blockDim.x, tid = threadIdx.x;
  const unsigned tmask = (1u << tbits) - 1u;
  auto slot0 = [&](int x) { return (unsigned)(((uint32_t)x * 2654435761u) >> (32 - tbits)) & tmask; };
  for (unsigned h = tid; h <= tmask; h += nt) table[h] = -1;
  __syncthreads();
  for (int j = tid; j < E; j += nt) {
    unsigned h = slot0(r[j]);
    while (atomicCAS(&table[h], -1, j) != -1) h = (h + 1) & tmask;
  }
  __syncthreads();
  int chain = 0;
  for (int j = tid; j < E; j += nt) {
    const int rj = r[j];
    int lp = -1, lvj = -1, later = 1;
    for (unsigned h = slot0(j);; h = (h + 1) & tmask) {      // steps i with r_i = j
      const int i = table[h];
      if (i < 0) break;
      if (r[i] == j && i < j && i > lp) lp = i;
    }
    for (unsigned h = slot0(rj);; h = (h + 1) & tmask) {     // steps i with r_i = r_j
      const int i = table[h];
      if (i < 0) break;
      if (r[i] == rj) {
        if (i < j && i > lvj) lvj = i;
        if (i > j) later = 0;
      }
    }
    par[j] = lp >= 0 ? lp : j;
    lv[j] = lvj;
    last_writer[j] = later;
    chain |= lp >= 0;
  }
  // Pointer jumping: after ceil(log2 E) rounds par[j] is the root of j's chain.
  int* src = par;
  int* dst = par2;
  if (__syncthreads_or(chain)) {
    for (int span = 1; span < E; span <<= 1) {
      for (int j = tid; j < E; j += nt) dst[j] = src[src[j]];
      __syncthreads();
      int* t = src; src = dst; dst = t;
    }
  }
  for (int j = tid; j < E; j += nt) pre[j] = base(src[j]);
  __syncthreads();
  for (int j = tid; j < E; j += nt) {
    const int rj = r[j];
    taken[j] = (rj == j) ? pre[j] : (lv[j] >= 0 ? pre[lv[j]] : base(rj));
  }
  __syncthreads();
}

// ------------------------------------------------------------------ kernels
__global__ void init_meta_kernel(int32_t* seen, long long* sample_id, int64_t C,
                                 unsigned long long* hist, ResCounters* ctr) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < C) {
    seen[i] = -1;
    sample_id[i] = -1;
  }
  if (i < kHistLen) hist[i] = 0;
  if (i < (int64_t)(sizeof(ResCounters) / sizeof(long long)))
    reinterpret_cast<long long*>(ctr)[i] = 0;
}

// Seen slots per tile of kTile slots: tile_cnt[t] = #{s in tile t : seen[s] >= 1}.
// grid = number of tiles, 256 threads x 4 slots.
__global__ __launch_bounds__(256) void seen_tile_count_kernel(const int32_t* __restrict__ seen, int64_t C,
                                                              int32_t* __restrict__ tile_cnt) {
  __shared__ int red[4];
  const int64_t s0 = (int64_t)blockIdx.x * kTile + threadIdx.x * 4;
  int c = 0;
  if (s0 + 3 < C) {
    const int4 v = *reinterpret_cast<const int4*>(seen + s0);
    c = (v.x >= 1) + (v.y >= 1) + (v.z >= 1) + (v.w >= 1);
  } else {
    for (int i = 0; i < 4; ++i) c += (s0 + i < C) && seen[s0 + i] >= 1;
  }
  for (int off = 32; off > 0; off >>= 1) c += __shfl_xor(c, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) tile_cnt[blockIdx.x] = red[0] + red[1] + red[2] + red[3];
}

// Put, metadata decisions.  One block.  a = min(k, C - U) rows are accepted;
// the first F = min(a, C - N) go to free slots N.., the other E = a - F
// replace seen samples chosen by a partial Fisher-Yates over the ascending
// list of seen slots (Philox kind 2, j = replacement index, range S - j).
// This kernel resolves the shuffle on *positions* of that list; the slots
// are found by put_victim_kernel from the tile prefix sums written here, and
// the per-slot metadata is written by put_copy_kernel.  `may_evict` is 0 when
// the host knows N + k <= C (then E = 0 and the tile counts were not made).
__global__ __launch_bounds__(kAssignThreads) void put_assign_kernel(
    int64_t k, uint64_t ticket, uint64_t seed, int64_t C, int may_evict, const int32_t* __restrict__ tile_cnt,
    int64_t ntiles, int32_t* __restrict__ tile_off, int32_t* __restrict__ victim_pos,
    int32_t* __restrict__ put_slots, ResCounters* __restrict__ ctr, long long* __restrict__ accepted_out) {
  // the shuffle's arrays of max(k, 1) ints and its table in dynamic LDS
  // (sized by the launch, so a small put does not hold a CU's LDS)
  extern __shared__ int s_dyn[];
  const int64_t cap = k > 0 ? k : 1;
  int *s_r = s_dyn, *s_par = s_r + cap, *s_par2 = s_par + cap, *s_lv = s_par2 + cap, *s_pre = s_lv + cap,
      *s_taken = s_pre + cap, *s_last = s_taken + cap, *s_tab = s_last + cap;
  const int tbits = shuffle_table_bits(cap);
  __shared__ int s_wave[kAssignThreads / 64];
  __shared__ int s_total;

  const long long U = ctr->U, S = ctr->S, N = ctr->N, base_id = ctr->next_sample_id;
  const long long a = min((long long)k, (long long)C - U);
  const long long F = min(a, (long long)C - N);
  const long long E = may_evict ? a - F : 0;
  const int tid = threadIdx.x, nt = blockDim.x;

  for (long long i = tid; i < F; i += nt) put_slots[i] = (int32_t)(N + i);
  for (long long j = tid; j < E; j += nt) put_slots[F + j] = -1;   // filled by put_victim_kernel

  if (E > 0) {
    // exclusive prefix sums of the tile counts (tile_off[ntiles] = S)
    int carry = 0;
    for (int64_t t0 = 0; t0 < ntiles; t0 += nt) {
      const int64_t t = t0 + tid;
      const int c = t < ntiles ? tile_cnt[t] : 0;
      const int off = block_exclusive_scan<kAssignThreads>(c, s_wave, &s_total);
      if (t < ntiles) tile_off[t] = carry + off;
      carry += s_total;
      __syncthreads();
    }
    if (tid == 0) tile_off[ntiles] = carry;
    for (long long j = tid; j < E; j += nt) {
      const uint64_t w = draw_word(seed, (uint64_t)j, ticket, kKindEvict);
      s_r[j] = (int)(j + (long long)range_map(w, (uint64_t)(S - j)));
    }
    __syncthreads();
    resolve_partial_shuffle((int)E, s_r, [](int p) { return p; }, s_tab, tbits, s_par, s_par2, s_lv, s_pre, s_taken,
                            s_last);
    for (long long j = tid; j < E; j += nt) victim_pos[j] = s_taken[j];
  }
  __syncthreads();
  if (tid == 0) {
    ctr->U = U + a;
    ctr->S = S - E;
    ctr->N = N + F;
    ctr->total_put += a;
    ctr->total_evicted += E;
    ctr->next_sample_id = base_id + a;
    ctr->last_accepted = a;
    ctr->last_free = F;
    ctr->last_evicted = E;
    ctr->last_base_id = base_id;
    if (accepted_out) *accepted_out = a;
  }
}

// Slot of each victim: position p of the ascending list of seen slots lies in
// the tile t with tile_off[t] <= p < tile_off[t + 1]; the rank p - tile_off[t]
// is found by one wavefront over the tile's seen counts.  Reads metadata only.
// grid = k blocks of 64 threads (block j handles victim j < E).
__global__ __launch_bounds__(64) void put_victim_kernel(const int32_t* __restrict__ seen, int64_t C,
                                                        const int32_t* __restrict__ tile_off, int64_t ntiles,
                                                        const int32_t* __restrict__ victim_pos,
                                                        int32_t* __restrict__ put_slots,
                                                        const ResCounters* __restrict__ ctr) {
  const int64_t j = blockIdx.x;
  if (j >= ctr->last_evicted) return;
  const int lane = threadIdx.x;
  const int p = victim_pos[j];
  // last tile whose offset is <= p (offsets are non-decreasing)
  int64_t tile = 0;
  for (int64_t b0 = 0; b0 < ntiles; b0 += 64) {
    const int64_t t = b0 + lane;
    const int v = t < ntiles ? tile_off[t] : 0x7fffffff;
    const uint64_t m = __ballot(v <= p);
    if (m == 0) break;
    tile = b0 + 63 - __clzll((long long)m);
    if (m != ~0ull) break;
  }
  const int rank = p - tile_off[tile];
  const int64_t s0 = tile * kTile + (int64_t)lane * (kTile / 64);
  int c = 0;
  for (int i = 0; i < kTile / 64; ++i) c += (s0 + i < C) && seen[s0 + i] >= 1;
  int incl = c;
  for (int off = 1; off < 64; off <<= 1) {
    const int t = __shfl_up(incl, off, 64);
    if (lane >= off) incl += t;
  }
  const int excl = incl - c;
  if (rank >= excl && rank < incl) {
    int want = rank - excl;
    for (int i = 0; i < kTile / 64; ++i) {
      if ((s0 + i < C) && seen[s0 + i] >= 1) {
        if (want == 0) {
          put_slots[ctr->last_free + j] = (int32_t)(s0 + i);
          break;
        }
        --want;
      }
    }
  }
}

// Put, metadata decisions in one launch, for reservoirs of up to
// kFusedMaxC slots and puts of up to kFusedMaxPut rows: the decisions of
// put_assign_kernel, with the ascending list of seen slots indexed inside the
// block instead of by seen_tile_count_kernel and put_victim_kernel.  The
// block reads the seen counts 256 slots per wavefront load (lane l: slots
// 4l .. 4l + 3 of the chunk) and keeps, per chunk c, four ballot masks
// (mask[c][i] bit l: slot 256c + 4l + i is seen) and the chunk's count; an
// exclusive scan of the counts gives the list position of each chunk's first
// seen slot.  Victim position p then maps to its chunk by binary search over
// those offsets, to its lane by binary search over the per-lane prefix counts
// of the chunk, and to the slot within the lane's four.  Same victims as the
// three-kernel path (same draws, same ascending order of seen slots).
constexpr int64_t kFusedMaxC = 262144;     // <= kAssignThreads chunks of 256 slots
constexpr int64_t kFusedMaxPut = 1024;
__global__ __launch_bounds__(kAssignThreads) void put_assign_fused_kernel(
    int64_t k, uint64_t ticket, uint64_t seed, int64_t C, int may_evict, const int32_t* __restrict__ seen,
    int32_t* __restrict__ put_slots, ResCounters* __restrict__ ctr, long long* __restrict__ accepted_out) {
  // dynamic LDS: the shuffle's arrays of max(k, 1) ints and its table, then
  // per chunk four 64-bit masks and (one more than the chunks) offsets
  extern __shared__ int s_dyn[];
  const int64_t cap = k > 0 ? k : 1;
  const int nchunks = (int)((C + 255) / 256);
  int *s_r = s_dyn, *s_par = s_r + cap, *s_par2 = s_par + cap, *s_lv = s_par2 + cap, *s_pre = s_lv + cap,
      *s_taken = s_pre + cap, *s_last = s_taken + cap, *s_tab = s_last + cap;
  const int tbits = shuffle_table_bits(cap);
  unsigned long long* s_mask = reinterpret_cast<unsigned long long*>(s_dyn + ((shuffle_lds_ints(cap) + 1) & ~1LL));
  int* s_off = reinterpret_cast<int*>(s_mask + 4 * (int64_t)nchunks);
  __shared__ int s_wave[kAssignThreads / 64];
  __shared__ int s_total;

  const long long U = ctr->U, S = ctr->S, N = ctr->N, base_id = ctr->next_sample_id;
  const long long a = min((long long)k, (long long)C - U);
  const long long F = min(a, (long long)C - N);
  const long long E = may_evict ? a - F : 0;
  const int tid = threadIdx.x, nt = blockDim.x, lane = tid & 63, wid = tid >> 6;

  for (long long i = tid; i < F; i += nt) put_slots[i] = (int32_t)(N + i);

  if (E > 0) {
    // seen masks: wavefront wid takes chunks wid, wid + 16, ...; eight
    // 16-byte loads in flight per lane, issued without branches (a load whose
    // first slot is past the end reads slot 0, and slots past the end are
    // masked; the seen array is allocated with 16 bytes to spare, so a load
    // that starts below C stays inside it)
    constexpr int B = 8;
    for (int c0 = wid; c0 < nchunks; c0 += B * (kAssignThreads / 64)) {
      int4 v[B];
#pragma unroll
      for (int u = 0; u < B; ++u) {
        const int64_t s0 = (int64_t)(c0 + u * (kAssignThreads / 64)) * 256 + 4 * lane;
        v[u] = *reinterpret_cast<const int4*>(seen + (s0 < C ? s0 : 0));
      }
#pragma unroll
      for (int u = 0; u < B; ++u) {
        const int c = c0 + u * (kAssignThreads / 64);
        const int64_t s0 = (int64_t)c * 256 + 4 * lane;
        const unsigned long long m0 = __ballot(s0 < C && v[u].x >= 1), m1 = __ballot(s0 + 1 < C && v[u].y >= 1),
                                 m2 = __ballot(s0 + 2 < C && v[u].z >= 1), m3 = __ballot(s0 + 3 < C && v[u].w >= 1);
        if (c < nchunks && lane == 0) {
          s_mask[4 * c + 0] = m0;
          s_mask[4 * c + 1] = m1;
          s_mask[4 * c + 2] = m2;
          s_mask[4 * c + 3] = m3;
          s_off[c] = __popcll(m0) + __popcll(m1) + __popcll(m2) + __popcll(m3);
        }
      }
    }
    __syncthreads();
    // exclusive offsets of the chunks (s_off[nchunks] = S)
    {
      const int cnt = tid < nchunks ? s_off[tid] : 0;
      __syncthreads();
      const int off = block_exclusive_scan<kAssignThreads>(cnt, s_wave, &s_total);
      if (tid < nchunks) s_off[tid] = off;
      if (tid == 0) s_off[nchunks] = s_total;
      __syncthreads();
    }
    for (long long j = tid; j < E; j += nt) {
      const uint64_t w = draw_word(seed, (uint64_t)j, ticket, kKindEvict);
      s_r[j] = (int)(j + (long long)range_map(w, (uint64_t)(S - j)));
    }
    __syncthreads();
    resolve_partial_shuffle((int)E, s_r, [](int p) { return p; }, s_tab, tbits, s_par, s_par2, s_lv, s_pre, s_taken,
                            s_last);
    for (long long j = tid; j < E; j += nt) {
      const int p = s_taken[j];
      // chunk: last c with s_off[c] <= p
      int lo = 0, hi = nchunks - 1;
      while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if (s_off[mid] <= p) lo = mid;
        else hi = mid - 1;
      }
      const int c = lo;
      const unsigned long long* m = s_mask + 4 * c;
      int rank = p - s_off[c];
      // lane: last l with (seen slots of lanes < l) <= rank
      auto below = [&](int l) {
        const unsigned long long lowm = l >= 64 ? ~0ull : ((1ull << l) - 1);
        return __popcll(m[0] & lowm) + __popcll(m[1] & lowm) + __popcll(m[2] & lowm) + __popcll(m[3] & lowm);
      };
      int llo = 0, lhi = 63;
      while (llo < lhi) {
        const int mid = (llo + lhi + 1) >> 1;
        if (below(mid) <= rank) llo = mid;
        else lhi = mid - 1;
      }
      rank -= below(llo);
      int slot = -1;
      for (int i = 0; i < 4; ++i)
        if ((m[i] >> llo) & 1ull) {
          if (rank == 0) {
            slot = c * 256 + 4 * llo + i;
            break;
          }
          --rank;
        }
      put_slots[F + j] = slot;
    }
  }
  __syncthreads();
  if (tid == 0) {
    ctr->U = U + a;
    ctr->S = S - E;
    ctr->N = N + F;
    ctr->total_put += a;
    ctr->total_evicted += E;
    ctr->next_sample_id = base_id + a;
    ctr->last_accepted = a;
    ctr->last_free = F;
    ctr->last_evicted = E;
    ctr->last_base_id = base_id;
    if (accepted_out) *accepted_out = a;
  }
}

constexpr int kCopyThreads = 256;
constexpr int kCopyVecPerThread = 4;
constexpr int64_t kCopySeg = (int64_t)kCopyThreads * kCopyVecPerThread * 4;  // floats per block

// Copy one row segment: dst[0..n) = src[0..n), float4 granules when aligned.
template <bool kNtLoad, bool kNtStore>
__device__ __forceinline__ void copy_segment(float* __restrict__ dst, const float* __restrict__ src,
                                             int64_t n, bool vec_ok) {
  const int t = threadIdx.x;
  if (vec_ok) {
    const int64_t n4 = n >> 2;
    const f32x4* s4 = reinterpret_cast<const f32x4*>(src);
    f32x4* d4 = reinterpret_cast<f32x4*>(dst);
    f32x4 v[kCopyVecPerThread];
#pragma unroll
    for (int u = 0; u < kCopyVecPerThread; ++u) {
      const int64_t i = (int64_t)u * kCopyThreads + t;
      if (i < n4) v[u] = kNtLoad ? __builtin_nontemporal_load(s4 + i) : s4[i];
    }
#pragma unroll
    for (int u = 0; u < kCopyVecPerThread; ++u) {
      const int64_t i = (int64_t)u * kCopyThreads + t;
      if (i < n4) {
        if (kNtStore) __builtin_nontemporal_store(v[u], d4 + i);
        else d4[i] = v[u];
      }
    }
    for (int64_t i = (n4 << 2) + t; i < n; i += kCopyThreads) dst[i] = src[i];
  } else {
    for (int64_t i = t; i < n; i += kCopyThreads) dst[i] = src[i];
  }
}

// Put, data half: row i < a of the chunk goes to slot put_slots[i].
// grid = k rows x `segs` segments per row, flattened (row-major).
__global__ __launch_bounds__(kCopyThreads) void put_copy_kernel(
    const float* __restrict__ x, int64_t ldx, const float* __restrict__ u, int64_t ldu,
    const int32_t* __restrict__ put_slots, const ResCounters* __restrict__ ctr,
    float* __restrict__ xslab, int64_t ldxs, float* __restrict__ uslab, int64_t ldus, int64_t x_dim,
    int64_t u_dim, int64_t segs, int vec_ok, int32_t* __restrict__ seen, long long* __restrict__ sample_id,
    unsigned long long* __restrict__ hist, int64_t C) {
  const int64_t row = (int64_t)blockIdx.x / segs, seg = (int64_t)blockIdx.x % segs;
  if (row >= ctr->last_accepted) return;
  const int64_t slot = put_slots[row];
  if (slot < 0 || slot >= C) return;   // never expected: every accepted row has a slot
  if (seg == 0 && threadIdx.x == 0) {
    // the slot's new sample: unseen, next id; a replaced seen sample is counted
    if (row >= ctr->last_free) atomicAdd(&hist[min(seen[slot], kHistLen - 1)], 1ull);
    seen[slot] = 0;
    sample_id[slot] = ctr->last_base_id + row;
  }
  const int64_t seg0 = seg * kCopySeg;
  const int64_t n = min(kCopySeg, u_dim - seg0);
  copy_segment<true, true>(uslab + slot * ldus + seg0, u + row * ldu + seg0, n, vec_ok != 0);
  if (seg == 0)
    for (int64_t c = threadIdx.x; c < x_dim; c += kCopyThreads)
      xslab[slot * ldxs + c] = x ? x[row * ldx + c] : 0.0f;
}

// Batch draw, normal phase: draw j picks slot floor(w_j N / 2^64), with
// replacement; a first draw turns the slot from unseen to seen.
__global__ void select_kernel(uint64_t seed, uint64_t ticket, int64_t N, int64_t b,
                              int32_t* __restrict__ slots, int32_t* __restrict__ seen,
                              ResCounters* __restrict__ ctr) {
  const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (j == 0) atomic_add_ll(&ctr->total_draws, b);
  if (j >= b) return;
  const uint64_t w = draw_word(seed, (uint64_t)j, ticket, kKindSample);
  const int32_t slot = (int32_t)range_map(w, (uint64_t)N);
  slots[j] = slot;
  const int old = atomicAdd(&seen[slot], 1);
  if (old == 0) {
    atomic_add_ll(&ctr->U, -1);
    atomic_add_ll(&ctr->S, 1);
  }
}

// Batch that takes its samples out of the list occ (ring of C positions from
// occ_base, N entries): the Reservoir after reception ends and FIRO draw
// bb distinct positions by partial Fisher-Yates (shuffle = 1: step j swaps
// positions j and j + floor(w_j (N - j) / 2^64), w_j = Philox(seed; j,
// ticket, 1), and takes position j); FIFO takes the first bb (shuffle = 0).
// The shuffled positions that stay in the list are written back, the taken
// slots are pushed on the free queue from position free_tail, and their
// metadata cleared.  One block.
__global__ __launch_bounds__(kAssignThreads) void list_take_kernel(
    uint64_t seed, uint64_t ticket, int64_t N, int64_t bb, int shuffle, int64_t occ_base, int64_t C,
    int32_t* __restrict__ occ, int32_t* __restrict__ free_q, int64_t free_tail, int32_t* __restrict__ slots,
    int32_t* __restrict__ seen, long long* __restrict__ sample_id, unsigned long long* __restrict__ hist,
    ResCounters* __restrict__ ctr) {
  // the shuffle's arrays of max(bb, 1) ints and its table in dynamic LDS, sized by the launch
  extern __shared__ int s_dyn[];
  const int64_t cap = bb > 0 ? bb : 1;
  int *s_r = s_dyn, *s_par = s_r + cap, *s_par2 = s_par + cap, *s_lv = s_par2 + cap, *s_pre = s_lv + cap,
      *s_taken = s_pre + cap, *s_last = s_taken + cap, *s_tab = s_last + cap;
  const int tbits = shuffle_table_bits(cap);
  __shared__ long long s_dU, s_dS;
  const int tid = threadIdx.x, nt = blockDim.x;
  auto pos = [&](int64_t p) { return (occ_base + p) % C; };
  if (tid == 0) { s_dU = 0; s_dS = 0; }
  if (shuffle) {
    for (long long j = tid; j < bb; j += nt) {
      const uint64_t w = draw_word(seed, (uint64_t)j, ticket, kKindSample);
      s_r[j] = (int)(j + (long long)range_map(w, (uint64_t)(N - j)));
    }
    __syncthreads();
    resolve_partial_shuffle((int)bb, s_r, [&](int p) { return (int)occ[pos(p)]; }, s_tab, tbits, s_par, s_par2,
                            s_lv, s_pre, s_taken, s_last);
    // Persist the shuffle for positions that stay in the list.
    for (long long j = tid; j < bb; j += nt)
      if (s_r[j] >= bb && s_last[j]) occ[pos(s_r[j])] = s_pre[j];
  } else {
    for (long long j = tid; j < bb; j += nt) s_taken[j] = occ[pos(j)];
  }
  __syncthreads();
  for (long long j = tid; j < bb; j += nt) {
    const int slot = s_taken[j];
    slots[j] = slot;
    free_q[(free_tail + j) % C] = slot;
    const int c = seen[slot] + 1;
    atomicAdd(&hist[min(c, kHistLen - 1)], 1ull);
    if (c == 1) atomicAdd((unsigned long long*)&s_dU, 1ull);
    else atomicAdd((unsigned long long*)&s_dS, 1ull);
    seen[slot] = -1;
    sample_id[slot] = -1;
  }
  __syncthreads();
  if (tid == 0) {
    ctr->U -= s_dU;
    ctr->S -= s_dS;
    ctr->N -= bb;
    ctr->total_deleted += bb;
    ctr->total_draws += bb;
  }
}

// FIFO / FIRO put, metadata decisions: the a = min(k, C - N) accepted rows
// take the slots at the head of the free queue and are appended to the list.
// a and every ring position are known on the host.
__global__ void list_put_kernel(int64_t a, int64_t N, int64_t occ_base, int64_t free_head, int64_t C,
                                const int32_t* __restrict__ free_q, int32_t* __restrict__ occ,
                                int32_t* __restrict__ put_slots, ResCounters* __restrict__ ctr,
                                long long* __restrict__ accepted_out) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < a) {
    const int32_t slot = free_q[(free_head + i) % C];
    put_slots[i] = slot;
    occ[(occ_base + N + i) % C] = slot;
  }
  if (i == 0) {
    const long long base_id = ctr->next_sample_id;
    ctr->U += a;
    ctr->N += a;
    ctr->total_put += a;
    ctr->next_sample_id = base_id + a;
    ctr->last_accepted = a;
    ctr->last_free = a;     // no row replaces a stored sample
    ctr->last_evicted = 0;
    ctr->last_base_id = base_id;
    if (accepted_out) *accepted_out = a;
  }
}

__global__ void iota_kernel(int32_t* occ, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) occ[i] = (int32_t)i;
}

// Gather rows of the drawn slots into the caller's batch buffers.
// grid = b rows x `segs` segments per row, flattened (row-major).
__global__ __launch_bounds__(kCopyThreads) void gather_kernel(
    const int32_t* __restrict__ slots, const float* __restrict__ xslab, int64_t ldxs,
    const float* __restrict__ uslab, int64_t ldus, float* __restrict__ x_out, int64_t ldxo,
    float* __restrict__ u_out, int64_t lduo, int64_t x_dim, int64_t u_dim, int64_t segs, int vec_ok) {
  const int64_t row = (int64_t)blockIdx.x / segs, seg = (int64_t)blockIdx.x % segs;
  const int64_t slot = slots[row];
  const int64_t seg0 = seg * kCopySeg;
  if (u_out) {
    const int64_t n = min(kCopySeg, u_dim - seg0);
    copy_segment<true, false>(u_out + row * lduo + seg0, uslab + slot * ldus + seg0, n, vec_ok != 0);
  }
  if (x_out && seg == 0)
    for (int64_t c = threadIdx.x; c < x_dim; c += kCopyThreads)
      x_out[row * ldxo + c] = xslab[slot * ldxs + c];
}

// Gather of the input rows alone (the field rows are read in place by the
// train step): one thread per copied value.  grid = ceil(b x_dim / 256).
__global__ __launch_bounds__(256) void gather_x_kernel(const int32_t* __restrict__ slots,
                                                       const float* __restrict__ xslab, int64_t ldxs,
                                                       float* __restrict__ x_out, int64_t ldxo, int64_t x_dim,
                                                       int64_t b) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= b * x_dim) return;
  const int64_t row = i / x_dim, c = i % x_dim;
  x_out[row * ldxo + c] = xslab[(int64_t)slots[row] * ldxs + c];
}

}  // namespace ot

// ===================================================================== host side
using ot::ResCounters;

struct ot_reservoir {
  int device = 0;
  ot::ResSeq seq;            // policy, C, T and the host-known state of the call sequence
  int64_t x_dim = 0, u_dim = 0, ldxs = 0, ldus = 0;
  uint64_t seed = 0;
  float* xslab = nullptr;
  float* uslab = nullptr;
  int32_t* seen = nullptr;
  long long* sample_id = nullptr;
  int32_t* occ = nullptr;
  int32_t* free_q = nullptr;   // FIFO / FIRO: ring of free slots
  int32_t* put_slots = nullptr;
  int32_t* tile_cnt = nullptr;
  int32_t* tile_off = nullptr;
  int32_t* victim_pos = nullptr;
  int64_t ntiles = 0;
  unsigned long long* hist = nullptr;
  ResCounters* ctr = nullptr;
  hipStream_t stream = nullptr;
  bool own_stream = false;
  hipEvent_t ev_in = nullptr, ev_out = nullptr;
  std::mutex mu;             // guards seq and the timer; held for the whole of every call
  ot::PhaseTimer timer;
};

namespace {

void free_reservoir(ot_reservoir* r) {
  if (!r) return;
  if (r->stream) (void)hipStreamSynchronize(r->stream);
  r->timer.release();
  (void)hipFree(r->xslab);
  (void)hipFree(r->uslab);
  (void)hipFree(r->seen);
  (void)hipFree(r->sample_id);
  (void)hipFree(r->occ);
  (void)hipFree(r->free_q);
  (void)hipFree(r->put_slots);
  (void)hipFree(r->tile_cnt);
  (void)hipFree(r->tile_off);
  (void)hipFree(r->victim_pos);
  (void)hipFree(r->hist);
  (void)hipFree(r->ctr);
  if (r->ev_in) (void)hipEventDestroy(r->ev_in);
  if (r->ev_out) (void)hipEventDestroy(r->ev_out);
  if (r->own_stream && r->stream) (void)hipStreamDestroy(r->stream);
  delete r;
}

template <class T>
int dev_alloc(T** p, size_t count) {
  hipError_t e = hipMalloc(reinterpret_cast<void**>(p), count * sizeof(T) + 16);
  if (e != hipSuccess) {
    (void)hipGetLastError();
    return ot::set_error(OT_E_NOMEM, "hipMalloc of %zu bytes failed: %s", count * sizeof(T),
                         hipGetErrorString(e));
  }
  return OT_OK;
}

// Order the reservoir's stream after the caller's work.
int enter(ot_reservoir* r, hipStream_t caller) {
  if (caller == r->stream) return OT_OK;
  OT_HIP(hipEventRecord(r->ev_in, caller));
  OT_HIP(hipStreamWaitEvent(r->stream, r->ev_in, 0));
  return OT_OK;
}

// Order the caller's stream after the reservoir's work.
int leave(ot_reservoir* r, hipStream_t caller) {
  if (caller == r->stream) return OT_OK;
  OT_HIP(hipEventRecord(r->ev_out, r->stream));
  OT_HIP(hipStreamWaitEvent(caller, r->ev_out, 0));
  return OT_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Dynamic LDS of put_assign_fused_kernel: the shuffle's seven arrays of
// max(k, 1) ints (rounded to 8 bytes), four 64-bit masks per 256-slot chunk
// and one offset per chunk plus one.
unsigned fused_assign_lds(int64_t C, int64_t k) {
  const int64_t cap = std::max<int64_t>(k, 1);
  const int64_t nchunks = ot::ceil_div(C, 256);
  return (unsigned)(((ot::shuffle_lds_ints(cap) + 1) & ~1LL) * sizeof(int) +
                    4 * nchunks * sizeof(unsigned long long) + (nchunks + 1) * sizeof(int));
}

// Dynamic LDS of put_assign_kernel and list_take_kernel for up to n steps.
unsigned shuffle_lds(int64_t n) { return (unsigned)(ot::shuffle_lds_ints(std::max<int64_t>(n, 1)) * sizeof(int)); }

}  // namespace

extern "C" int reservoir_create(ot_reservoir** out, int64_t capacity, int64_t threshold,
                                int64_t x_dim, int64_t u_dim, uint64_t seed, int32_t policy,
                                void* order_stream) {
  ot::clear_error();
  OT_REQUIRE(out != nullptr, "reservoir_create: out is NULL");
  *out = nullptr;
  OT_REQUIRE(policy == OT_POLICY_RESERVOIR || policy == OT_POLICY_FIFO || policy == OT_POLICY_FIRO,
             "reservoir_create: unknown policy %d", (int)policy);
  OT_REQUIRE(capacity >= 1 && capacity <= 0x7fffffffLL, "reservoir_create: capacity %lld outside [1, 2^31-1]",
             (long long)capacity);
  OT_REQUIRE(threshold >= 0, "reservoir_create: threshold < 0");
  OT_REQUIRE(x_dim >= 1 && x_dim <= 4096, "reservoir_create: x_dim outside [1, 4096]");
  OT_REQUIRE(u_dim >= 1 && u_dim <= (1LL << 31), "reservoir_create: u_dim outside [1, 2^31]");
  ot_reservoir* r = new ot_reservoir();
  r->seq.policy = policy;
  r->seq.C = capacity;
  r->seq.T = threshold;
  r->x_dim = x_dim;
  r->u_dim = u_dim;
  r->ldxs = ot::round_up(x_dim, 4);
  r->ldus = ot::round_up(u_dim, 64);
  r->seed = seed;
  int rc = OT_OK;
  auto fail = [&](int code) {
    free_reservoir(r);
    return code;
  };
  if (hipGetDevice(&r->device) != hipSuccess) return fail(ot::set_error(OT_E_HIP, "hipGetDevice failed"));
  if ((rc = dev_alloc(&r->xslab, (size_t)capacity * r->ldxs))) return fail(rc);
  if ((rc = dev_alloc(&r->uslab, (size_t)capacity * r->ldus))) return fail(rc);
  if ((rc = dev_alloc(&r->seen, (size_t)capacity))) return fail(rc);
  if ((rc = dev_alloc(&r->sample_id, (size_t)capacity))) return fail(rc);
  if ((rc = dev_alloc(&r->occ, (size_t)capacity))) return fail(rc);
  if ((rc = dev_alloc(&r->free_q, (size_t)capacity))) return fail(rc);
  if ((rc = dev_alloc(&r->put_slots, (size_t)ot::kMaxPut))) return fail(rc);
  r->ntiles = ot::ceil_div(capacity, ot::kTile);
  if ((rc = dev_alloc(&r->tile_cnt, (size_t)r->ntiles))) return fail(rc);
  if ((rc = dev_alloc(&r->tile_off, (size_t)r->ntiles + 1))) return fail(rc);
  if ((rc = dev_alloc(&r->victim_pos, (size_t)ot::kMaxPut))) return fail(rc);
  if ((rc = dev_alloc(&r->hist, (size_t)ot::kHistLen))) return fail(rc);
  if ((rc = dev_alloc(&r->ctr, 1))) return fail(rc);
  if (order_stream) {
    r->stream = static_cast<hipStream_t>(order_stream);
  } else {
    if (hipStreamCreateWithFlags(&r->stream, hipStreamNonBlocking) != hipSuccess)
      return fail(ot::set_error(OT_E_HIP, "hipStreamCreate failed"));
    r->own_stream = true;
  }
  {
    // the assignment and take kernels size their LDS per call (the shuffle's arrays and table for the largest call)
    const int max_dyn = (int)shuffle_lds(std::max(ot::kMaxPut, ot::kMaxDrainBatch));
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(&ot::put_assign_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, max_dyn) != hipSuccess ||
        hipFuncSetAttribute(reinterpret_cast<const void*>(&ot::put_assign_fused_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)fused_assign_lds(ot::kFusedMaxC, ot::kFusedMaxPut)) != hipSuccess ||
        hipFuncSetAttribute(reinterpret_cast<const void*>(&ot::list_take_kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, max_dyn) != hipSuccess)
      return fail(ot::set_error(OT_E_HIP, "hipFuncSetAttribute (dynamic LDS) failed"));
  }
  if (hipEventCreateWithFlags(&r->ev_in, hipEventDisableTiming) != hipSuccess ||
      hipEventCreateWithFlags(&r->ev_out, hipEventDisableTiming) != hipSuccess)
    return fail(ot::set_error(OT_E_HIP, "hipEventCreate failed"));
  const int64_t n_init = std::max<int64_t>(capacity, 64);
  hipLaunchKernelGGL(ot::init_meta_kernel, dim3((unsigned)ot::ceil_div(n_init, 256)), dim3(256), 0,
                     r->stream, r->seen, r->sample_id, capacity, r->hist, r->ctr);
  if (hipGetLastError() != hipSuccess) return fail(ot::set_error(OT_E_HIP, "init_meta_kernel launch failed"));
  if (policy != OT_POLICY_RESERVOIR) {   // every slot free, in slot order
    hipLaunchKernelGGL(ot::iota_kernel, dim3((unsigned)ot::ceil_div(capacity, 256)), dim3(256), 0, r->stream,
                       r->free_q, capacity);
    if (hipGetLastError() != hipSuccess) return fail(ot::set_error(OT_E_HIP, "iota_kernel launch failed"));
  }
  if (hipStreamSynchronize(r->stream) != hipSuccess)
    return fail(ot::set_error(OT_E_HIP, "reservoir_create: stream synchronise failed"));
  *out = r;
  return OT_OK;
}

extern "C" int reservoir_put(ot_reservoir* r, const float* x, int64_t ldx, const float* u,
                             int64_t ldu, int64_t k, void* stream, int64_t* accepted_dev,
                             uint64_t* ticket_out) {
  ot::clear_error();
  OT_REQUIRE(r != nullptr, "reservoir_put: NULL reservoir");
  OT_REQUIRE(k >= 0 && k <= ot::kMaxPut, "reservoir_put: k=%lld outside [0, %lld]", (long long)k,
             (long long)ot::kMaxPut);
  if (k > 0) {
    OT_REQUIRE(u != nullptr, "reservoir_put: u is NULL");
    OT_REQUIRE(ldu >= r->u_dim, "reservoir_put: ldu < u_dim");
    OT_REQUIRE(x == nullptr || ldx >= r->x_dim, "reservoir_put: ldx < x_dim");
  }
  hipStream_t cs = static_cast<hipStream_t>(stream);
  std::lock_guard<std::mutex> lock(r->mu);
  if (ot::put_admit(r->seq) != OT_OK) return ot::set_error(OT_E_CLOSED, "reservoir_put: reception is over");
  // the ticket is taken only once the ordering stream waits for the caller:
  // a call that fails before enqueueing anything leaves the ticket sequence unchanged
  int rc = enter(r, cs);
  if (rc) return rc;
  const ot::PutCall pc = ot::put_commit(r->seq, k);
  const uint64_t ticket = pc.ticket;
  if (ticket_out) *ticket_out = ticket;
  ot::PhaseTimer& tm = r->timer;
  if (r->seq.policy != OT_POLICY_RESERVOIR) {
    // FIFO / FIRO: the accepted prefix and every ring position are host-known
    const int64_t a = pc.accepted;
    tm.mark(r->stream, OT_PH_PUT_ASSIGN, 0);
    hipLaunchKernelGGL(ot::list_put_kernel, dim3((unsigned)std::max<int64_t>(1, ot::ceil_div(a, 256))), dim3(256),
                       0, r->stream, a, pc.n_before, r->seq.occ_base, pc.free_head, r->seq.C, r->free_q, r->occ,
                       r->put_slots, r->ctr, reinterpret_cast<long long*>(accepted_dev));
    OT_LAUNCHED("list_put_kernel");
    tm.mark(r->stream, OT_PH_PUT_ASSIGN, 1);
    if (a > 0) {
      hipEvent_t t0, t1;
      tm.kernel_events(OT_PH_PUT_COPY, &t0, &t1);
      const int vec_ok = aligned16(u) && (ldu % 4 == 0);
      const int64_t segs = ot::ceil_div(r->u_dim, ot::kCopySeg);
      hipExtLaunchKernelGGL(ot::put_copy_kernel, dim3((unsigned)(segs * a)), dim3(ot::kCopyThreads), 0, r->stream,
                            t0, t1, 0, x, ldx, u, ldu, r->put_slots, (const ot::ResCounters*)r->ctr, r->xslab,
                            r->ldxs, r->uslab, r->ldus, r->x_dim, r->u_dim, segs, vec_ok, r->seen, r->sample_id,
                            r->hist, r->seq.C);
      OT_LAUNCHED("put_copy_kernel");
    }
    tm.next_call();
    return leave(r, cs);
  }
  tm.mark(r->stream, OT_PH_PUT_ASSIGN, 0);
  // Replacement is possible only if N + k > C (host-known N); only then are
  // the seen slots indexed.
  const int may_evict = pc.may_evict;
  if (r->seq.C <= ot::kFusedMaxC && k <= ot::kFusedMaxPut) {
    hipLaunchKernelGGL(ot::put_assign_fused_kernel, dim3(1), dim3(ot::kAssignThreads), fused_assign_lds(r->seq.C, k),
                       r->stream, k, ticket, r->seed, r->seq.C, may_evict, (const int32_t*)r->seen, r->put_slots, r->ctr,
                       reinterpret_cast<long long*>(accepted_dev));
    OT_LAUNCHED("put_assign_fused_kernel");
  } else {
  if (may_evict) {
    hipLaunchKernelGGL(ot::seen_tile_count_kernel, dim3((unsigned)r->ntiles), dim3(256), 0, r->stream, r->seen,
                       r->seq.C, r->tile_cnt);
    OT_LAUNCHED("seen_tile_count_kernel");
  }
  hipLaunchKernelGGL(ot::put_assign_kernel, dim3(1), dim3(ot::kAssignThreads),
                     shuffle_lds(k), r->stream, k, ticket, r->seed,
                     r->seq.C, may_evict, r->tile_cnt, r->ntiles, r->tile_off, r->victim_pos, r->put_slots, r->ctr,
                     reinterpret_cast<long long*>(accepted_dev));
  OT_LAUNCHED("put_assign_kernel");
  if (may_evict && k > 0) {
    hipLaunchKernelGGL(ot::put_victim_kernel, dim3((unsigned)k), dim3(64), 0, r->stream, r->seen, r->seq.C,
                       r->tile_off, r->ntiles, r->victim_pos, r->put_slots, r->ctr);
    OT_LAUNCHED("put_victim_kernel");
  }
  }
  tm.mark(r->stream, OT_PH_PUT_ASSIGN, 1);
  if (k > 0) {
    hipEvent_t t0, t1;
    tm.kernel_events(OT_PH_PUT_COPY, &t0, &t1);
    const int vec_ok = aligned16(u) && (ldu % 4 == 0);
    const int64_t segs = ot::ceil_div(r->u_dim, ot::kCopySeg);
    hipExtLaunchKernelGGL(ot::put_copy_kernel, dim3((unsigned)(segs * k)), dim3(ot::kCopyThreads), 0, r->stream, t0,
                          t1, 0, x, ldx, u, ldu, r->put_slots, (const ot::ResCounters*)r->ctr, r->xslab, r->ldxs,
                          r->uslab, r->ldus, r->x_dim, r->u_dim, segs, vec_ok, r->seen, r->sample_id, r->hist, r->seq.C);
    OT_LAUNCHED("put_copy_kernel");
  }
  tm.next_call();
  return leave(r, cs);
}

extern "C" int reservoir_sample_batch(ot_reservoir* r, int64_t b, void* stream, int32_t* slots,
                                      float* x_out, int64_t ldxo, float* u_out, int64_t lduo,
                                      int64_t* count_out, uint64_t* ticket_out) {
  ot::clear_error();
  if (count_out) *count_out = 0;
  OT_REQUIRE(r != nullptr, "reservoir_sample_batch: NULL reservoir");
  OT_REQUIRE(b >= 1 && b <= ot::kMaxBatch, "reservoir_sample_batch: b=%lld outside [1, %lld]", (long long)b,
             (long long)ot::kMaxBatch);
  OT_REQUIRE(slots != nullptr, "reservoir_sample_batch: slots is NULL");
  OT_REQUIRE(u_out == nullptr || lduo >= r->u_dim, "reservoir_sample_batch: lduo < u_dim");
  OT_REQUIRE(x_out == nullptr || ldxo >= r->x_dim, "reservoir_sample_batch: ldxo < x_dim");
  hipStream_t cs = static_cast<hipStream_t>(stream);
  const bool list_take = r->seq.policy != OT_POLICY_RESERVOIR;   // FIFO / FIRO take samples out
  if (list_take)
    OT_REQUIRE(b <= ot::kMaxDrainBatch, "reservoir_sample_batch: b=%lld above %lld for a FIFO / FIRO buffer",
               (long long)b, (long long)ot::kMaxDrainBatch);
  std::lock_guard<std::mutex> lock(r->mu);
  int64_t drawn = b;
  const int admit = ot::draw_admit(r->seq, b, &drawn);
  if (admit != OT_OK) return admit;
  if (r->seq.reception_over)
    OT_REQUIRE(b <= ot::kMaxDrainBatch, "reservoir_sample_batch: b=%lld above %lld while draining",
               (long long)b, (long long)ot::kMaxDrainBatch);
  int rc = enter(r, cs);
  if (rc) return rc;
  const ot::DrawCall dc = ot::draw_commit(r->seq, drawn);
  const uint64_t ticket = dc.ticket;
  if (ticket_out) *ticket_out = ticket;
  ot::PhaseTimer& tm = r->timer;
  tm.mark(r->stream, OT_PH_SELECT, 0);
  if (!dc.take) {
    hipLaunchKernelGGL(ot::select_kernel, dim3((unsigned)ot::ceil_div(b, 256)), dim3(256), 0, r->stream,
                       r->seed, ticket, dc.n_before, b, slots, r->seen, r->ctr);
    OT_LAUNCHED("select_kernel");
  } else {
    hipLaunchKernelGGL(ot::list_take_kernel, dim3(1), dim3(ot::kAssignThreads),
                       shuffle_lds(drawn), r->stream, r->seed, ticket,
                       dc.n_before, drawn, r->seq.policy == OT_POLICY_FIFO ? 0 : 1, dc.occ_base, r->seq.C, r->occ,
                       r->free_q, dc.free_tail, slots, r->seen, r->sample_id, r->hist, r->ctr);
    OT_LAUNCHED("list_take_kernel");
  }
  tm.mark(r->stream, OT_PH_SELECT, 1);
  if (x_out && !u_out) {
    hipEvent_t t0, t1;
    tm.kernel_events(OT_PH_GATHER, &t0, &t1);
    hipExtLaunchKernelGGL(ot::gather_x_kernel, dim3((unsigned)ot::ceil_div(drawn * r->x_dim, 256)), dim3(256), 0,
                          r->stream, t0, t1, 0, (const int32_t*)slots, (const float*)r->xslab, r->ldxs, x_out,
                          ldxo, r->x_dim, drawn);
    OT_LAUNCHED("gather_x_kernel");
  } else if (u_out) {
    hipEvent_t t0, t1;
    tm.kernel_events(OT_PH_GATHER, &t0, &t1);
    const int vec_ok = (u_out == nullptr) || (aligned16(u_out) && (lduo % 4 == 0));
    const int64_t segs = ot::ceil_div(r->u_dim, ot::kCopySeg);
    hipExtLaunchKernelGGL(ot::gather_kernel, dim3((unsigned)(segs * drawn)), dim3(ot::kCopyThreads), 0, r->stream,
                          t0, t1, 0, (const int32_t*)slots, (const float*)r->xslab, r->ldxs,
                          (const float*)r->uslab, r->ldus, x_out, ldxo, u_out, lduo, r->x_dim, r->u_dim, segs,
                          vec_ok);
    OT_LAUNCHED("gather_kernel");
  }
  tm.next_call();
  if (count_out) *count_out = drawn;
  return leave(r, cs);
}

extern "C" int reservoir_end_reception(ot_reservoir* r) {
  ot::clear_error();
  OT_REQUIRE(r != nullptr, "reservoir_end_reception: NULL reservoir");
  std::lock_guard<std::mutex> lock(r->mu);
  if (ot::end_commit(r->seq) != OT_OK) return ot::set_error(OT_E_STATE, "reservoir_end_reception: already over");
  if (r->seq.policy != OT_POLICY_RESERVOIR) return OT_OK;   // the list is already maintained
  if (r->seq.n_host > 0) {
    hipLaunchKernelGGL(ot::iota_kernel, dim3((unsigned)ot::ceil_div(r->seq.n_host, 256)), dim3(256), 0, r->stream,
                       r->occ, r->seq.n_host);
    OT_LAUNCHED("iota_kernel");
  }
  return OT_OK;
}

extern "C" int reservoir_slab(ot_reservoir* r, const float** x, int64_t* ldx, const float** u, int64_t* ldu) {
  ot::clear_error();
  OT_REQUIRE(r != nullptr, "reservoir_slab: NULL reservoir");
  if (x) *x = r->xslab;
  if (ldx) *ldx = r->ldxs;
  if (u) *u = r->uslab;
  if (ldu) *ldu = r->ldus;
  return OT_OK;
}

extern "C" int reservoir_stats(ot_reservoir* r, ot_reservoir_stats* out) {
  ot::clear_error();
  OT_REQUIRE(r != nullptr && out != nullptr, "reservoir_stats: NULL argument");
  std::lock_guard<std::mutex> lock(r->mu);
  OT_HIP(hipStreamSynchronize(r->stream));
  ResCounters c;
  OT_HIP(hipMemcpy(&c, r->ctr, sizeof c, hipMemcpyDeviceToHost));
  out->capacity = r->seq.C;
  out->threshold = r->seq.T;
  out->n = c.N;
  out->unseen = c.U;
  out->seen = c.S;
  out->total_put = c.total_put;
  out->total_evicted = c.total_evicted;
  out->total_deleted = c.total_deleted;
  out->total_draws = c.total_draws;
  out->next_ticket = (int64_t)r->seq.next_ticket;
  out->next_sample_id = c.next_sample_id;
  out->reception_over = r->seq.reception_over ? 1 : 0;
  out->hist_len = ot::kHistLen;
  out->policy = r->seq.policy;
  out->reserved = 0;
  return OT_OK;
}

extern "C" int reservoir_read_meta(ot_reservoir* r, int32_t* seen_count, int64_t* sample_id,
                                   int64_t* evict_hist) {
  ot::clear_error();
  OT_REQUIRE(r != nullptr, "reservoir_read_meta: NULL reservoir");
  std::lock_guard<std::mutex> lock(r->mu);
  OT_HIP(hipStreamSynchronize(r->stream));
  if (seen_count) OT_HIP(hipMemcpy(seen_count, r->seen, r->seq.C * sizeof(int32_t), hipMemcpyDeviceToHost));
  if (sample_id) OT_HIP(hipMemcpy(sample_id, r->sample_id, r->seq.C * sizeof(int64_t), hipMemcpyDeviceToHost));
  if (evict_hist)
    OT_HIP(hipMemcpy(evict_hist, r->hist, ot::kHistLen * sizeof(int64_t), hipMemcpyDeviceToHost));
  return OT_OK;
}

extern "C" int reservoir_read_rows(ot_reservoir* r, const int32_t* slots_host, int64_t n, float* x_host,
                                   float* u_host) {
  ot::clear_error();
  OT_REQUIRE(r != nullptr && slots_host != nullptr && n >= 0, "reservoir_read_rows: bad argument");
  for (int64_t i = 0; i < n; ++i)
    OT_REQUIRE(slots_host[i] >= 0 && slots_host[i] < r->seq.C, "reservoir_read_rows: slot %d out of range",
               (int)slots_host[i]);
  std::lock_guard<std::mutex> lock(r->mu);
  OT_HIP(hipStreamSynchronize(r->stream));
  for (int64_t i = 0; i < n; ++i) {
    const int64_t s = slots_host[i];
    if (x_host)
      OT_HIP(hipMemcpy(x_host + i * r->x_dim, r->xslab + s * r->ldxs, r->x_dim * sizeof(float),
                       hipMemcpyDeviceToHost));
    if (u_host)
      OT_HIP(hipMemcpy(u_host + i * r->u_dim, r->uslab + s * r->ldus, r->u_dim * sizeof(float),
                       hipMemcpyDeviceToHost));
  }
  return OT_OK;
}

// ------------------------------------------------------------------ checkpoint
// Blob layout (host memory, native byte order): magic "OTRESV1", then int64
// fields policy, C, T, x_dim, u_dim, seed, next_ticket, n_host, occ_base,
// free_head, reception_over, n_rows, hist_len; the device counter block; the
// eviction histogram (uint64[hist_len]); seen int32[C], sample_id int64[C],
// occ int32[C], free_q int32[C]; then the x_dim + u_dim fp32 values of every
// occupied slot in ascending slot order.
namespace {

constexpr char kResMagic[8] = {'O', 'T', 'R', 'E', 'S', 'V', '1', 0};
constexpr int64_t kResHeaderWords = 13;

int64_t res_blob_bytes(const ot_reservoir* r, int64_t n_rows) {
  return 8 + kResHeaderWords * 8 + (int64_t)sizeof(ResCounters) + ot::kHistLen * 8 + r->seq.C * (4 + 8 + 4 + 4) +
         n_rows * (r->x_dim + r->u_dim) * 4;
}

// Runs [first, last] of consecutive slots with seen >= 0, in ascending order.
template <class F>
int for_each_occupied_run(const std::vector<int32_t>& seen, F f) {
  const int64_t C = (int64_t)seen.size();
  int64_t row = 0;
  for (int64_t s0 = 0; s0 < C;) {
    if (seen[s0] < 0) { ++s0; continue; }
    int64_t s1 = s0;
    while (s1 + 1 < C && seen[s1 + 1] >= 0) ++s1;
    int rc = f(s0, s1 - s0 + 1, row);
    if (rc) return rc;
    row += s1 - s0 + 1;
    s0 = s1 + 1;
  }
  return OT_OK;
}

}  // namespace

extern "C" int reservoir_checkpoint_size(ot_reservoir* r, int64_t* bytes) {
  ot::clear_error();
  OT_REQUIRE(r != nullptr && bytes != nullptr, "reservoir_checkpoint_size: NULL argument");
  std::lock_guard<std::mutex> lock(r->mu);
  OT_HIP(hipStreamSynchronize(r->stream));
  ResCounters c;
  OT_HIP(hipMemcpy(&c, r->ctr, sizeof c, hipMemcpyDeviceToHost));
  *bytes = res_blob_bytes(r, c.N);
  return OT_OK;
}

extern "C" int reservoir_checkpoint(ot_reservoir* r, void* buf, int64_t bytes) {
  ot::clear_error();
  OT_REQUIRE(r != nullptr && buf != nullptr, "reservoir_checkpoint: NULL argument");
  std::lock_guard<std::mutex> lock(r->mu);
  OT_HIP(hipStreamSynchronize(r->stream));
  const int64_t C = r->seq.C;
  ResCounters c;
  std::vector<unsigned long long> hist(ot::kHistLen);
  std::vector<int32_t> seen(C), occ(C), freeq(C);
  std::vector<long long> ids(C);
  OT_HIP(hipMemcpy(&c, r->ctr, sizeof c, hipMemcpyDeviceToHost));
  OT_HIP(hipMemcpy(hist.data(), r->hist, ot::kHistLen * 8, hipMemcpyDeviceToHost));
  OT_HIP(hipMemcpy(seen.data(), r->seen, C * 4, hipMemcpyDeviceToHost));
  OT_HIP(hipMemcpy(ids.data(), r->sample_id, C * 8, hipMemcpyDeviceToHost));
  OT_HIP(hipMemcpy(occ.data(), r->occ, C * 4, hipMemcpyDeviceToHost));
  OT_HIP(hipMemcpy(freeq.data(), r->free_q, C * 4, hipMemcpyDeviceToHost));
  int64_t n_rows = 0;
  for (int32_t v : seen) n_rows += v >= 0;
  if (n_rows != c.N || n_rows != r->seq.n_host)
    return ot::set_error(OT_E_STATE, "reservoir_checkpoint: %lld occupied slots but N = %lld (host %lld)",
                         (long long)n_rows, (long long)c.N, (long long)r->seq.n_host);
  OT_REQUIRE(bytes >= res_blob_bytes(r, n_rows), "reservoir_checkpoint: buffer of %lld bytes, %lld needed",
             (long long)bytes, (long long)res_blob_bytes(r, n_rows));
  ot::BlobWriter w(buf, bytes);
  __builtin_memcpy(w.take(8), kResMagic, 8);
  for (int64_t v : {(int64_t)r->seq.policy, C, r->seq.T, r->x_dim, r->u_dim, (int64_t)r->seed, (int64_t)r->seq.next_ticket,
                    r->seq.n_host, r->seq.occ_base, r->seq.free_head, (int64_t)r->seq.reception_over, n_rows,
                    (int64_t)ot::kHistLen})
    w.put(v);
  w.put(c);
  __builtin_memcpy(w.take(ot::kHistLen * 8), hist.data(), ot::kHistLen * 8);
  __builtin_memcpy(w.take(C * 4), seen.data(), C * 4);
  __builtin_memcpy(w.take(C * 8), ids.data(), C * 8);
  __builtin_memcpy(w.take(C * 4), occ.data(), C * 4);
  __builtin_memcpy(w.take(C * 4), freeq.data(), C * 4);
  const int64_t row_bytes = (r->x_dim + r->u_dim) * 4;
  unsigned char* rows = w.take(n_rows * row_bytes);
  if (!w.good) return ot::set_error(OT_E_STATE, "reservoir_checkpoint: blob overrun");
  return for_each_occupied_run(seen, [&](int64_t s0, int64_t n, int64_t row) -> int {
    unsigned char* dst = rows + row * row_bytes;
    OT_HIP(hipMemcpy2D(dst, row_bytes, r->xslab + s0 * r->ldxs, r->ldxs * 4, r->x_dim * 4, n,
                       hipMemcpyDeviceToHost));
    OT_HIP(hipMemcpy2D(dst + r->x_dim * 4, row_bytes, r->uslab + s0 * r->ldus, r->ldus * 4, r->u_dim * 4, n,
                       hipMemcpyDeviceToHost));
    return OT_OK;
  });
}

extern "C" int reservoir_restore(ot_reservoir* r, const void* buf, int64_t bytes) {
  ot::clear_error();
  OT_REQUIRE(r != nullptr && buf != nullptr, "reservoir_restore: NULL argument");
  ot::BlobReader rd(buf, bytes);
  const unsigned char* magic = rd.take(8);
  OT_REQUIRE(magic != nullptr && __builtin_memcmp(magic, kResMagic, 8) == 0, "reservoir_restore: not a reservoir checkpoint");
  int64_t h[kResHeaderWords];
  for (int64_t& v : h) v = rd.get<int64_t>();
  const int64_t policy = h[0], C = h[1], T = h[2], x_dim = h[3], u_dim = h[4], n_host = h[7], occ_base = h[8],
                free_head = h[9], n_rows = h[11], hist_len = h[12];
  OT_REQUIRE(rd.good, "reservoir_restore: truncated header");
  OT_REQUIRE(policy == r->seq.policy && C == r->seq.C && x_dim == r->x_dim && u_dim == r->u_dim,
             "reservoir_restore: checkpoint of a different buffer (policy %lld, C %lld, x_dim %lld, u_dim %lld)",
             (long long)policy, (long long)C, (long long)x_dim, (long long)u_dim);
  OT_REQUIRE(hist_len == ot::kHistLen && T >= 0 && n_host >= 0 && n_host <= C && n_rows == n_host &&
                 occ_base >= 0 && occ_base < C && free_head >= 0 && free_head < C,
             "reservoir_restore: inconsistent checkpoint header");
  OT_REQUIRE(bytes >= res_blob_bytes(r, n_rows), "reservoir_restore: checkpoint truncated");
  const ResCounters c = rd.get<ResCounters>();
  const unsigned char* hist = rd.take(ot::kHistLen * 8);
  std::vector<int32_t> seen(C);
  __builtin_memcpy(seen.data(), rd.take(C * 4), C * 4);
  const unsigned char* ids = rd.take(C * 8);
  const unsigned char* occ = rd.take(C * 4);
  const unsigned char* freeq = rd.take(C * 4);
  const int64_t row_bytes = (x_dim + u_dim) * 4;
  const unsigned char* rows = rd.take(n_rows * row_bytes);
  OT_REQUIRE(rd.good, "reservoir_restore: checkpoint truncated");
  int64_t occupied = 0;
  for (int32_t v : seen) occupied += v >= 0;
  OT_REQUIRE(occupied == n_rows && c.N == n_rows, "reservoir_restore: inconsistent slot metadata");
  std::lock_guard<std::mutex> lock(r->mu);
  OT_HIP(hipStreamSynchronize(r->stream));
  OT_HIP(hipMemcpy(r->ctr, &c, sizeof c, hipMemcpyHostToDevice));
  OT_HIP(hipMemcpy(r->hist, hist, ot::kHistLen * 8, hipMemcpyHostToDevice));
  OT_HIP(hipMemcpy(r->seen, seen.data(), C * 4, hipMemcpyHostToDevice));
  OT_HIP(hipMemcpy(r->sample_id, ids, C * 8, hipMemcpyHostToDevice));
  OT_HIP(hipMemcpy(r->occ, occ, C * 4, hipMemcpyHostToDevice));
  OT_HIP(hipMemcpy(r->free_q, freeq, C * 4, hipMemcpyHostToDevice));
  int rc = for_each_occupied_run(seen, [&](int64_t s0, int64_t n, int64_t row) -> int {
    const unsigned char* src = rows + row * row_bytes;
    OT_HIP(hipMemcpy2D(r->xslab + s0 * r->ldxs, r->ldxs * 4, src, row_bytes, r->x_dim * 4, n,
                       hipMemcpyHostToDevice));
    OT_HIP(hipMemcpy2D(r->uslab + s0 * r->ldus, r->ldus * 4, src + r->x_dim * 4, row_bytes, r->u_dim * 4, n,
                       hipMemcpyHostToDevice));
    return OT_OK;
  });
  if (rc) return rc;
  r->seq.T = T;
  r->seed = (uint64_t)h[5];
  r->seq.next_ticket = (uint64_t)h[6];
  r->seq.n_host = n_host;
  r->seq.occ_base = occ_base;
  r->seq.free_head = free_head;
  r->seq.reception_over = h[10] != 0;
  return OT_OK;
}

extern "C" int reservoir_destroy(ot_reservoir* r) {
  ot::clear_error();
  if (!r) return OT_OK;
  free_reservoir(r);
  return OT_OK;
}

extern "C" int reservoir_timing_begin(ot_reservoir* r, uint32_t phase_mask, int64_t max_calls) {
  ot::clear_error();
  OT_REQUIRE(r != nullptr, "reservoir_timing_begin: NULL reservoir");
  OT_REQUIRE(phase_mask != 0 && phase_mask < (1u << OT_RESERVOIR_PHASES), "reservoir_timing_begin: bad mask");
  std::lock_guard<std::mutex> lock(r->mu);
  return r->timer.begin(phase_mask, OT_RESERVOIR_PHASES, max_calls);
}

extern "C" int reservoir_timing_end(ot_reservoir* r, double* ms_total, int64_t* count) {
  ot::clear_error();
  OT_REQUIRE(r != nullptr, "reservoir_timing_end: NULL reservoir");
  std::lock_guard<std::mutex> lock(r->mu);
  return r->timer.end(ms_total, count);
}
