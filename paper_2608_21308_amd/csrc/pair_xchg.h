// Several workgroups per unit: exchange of partial sums through global memory.
//
// For the widest fast-weight nets one unit's hidden columns are split between
// NS workgroups (NS = 2 to 8; ranks 0 .. NS-1 of a group), each holding its
// share of the state in registers.  Contractions over the hidden index then
// give each rank a partial C x d sum that the others need; the ranks swap
// these through a small global buffer and a flag per rank.  Every rank adds
// the NS partials in rank order, so all ranks see bitwise identical sums.
//
// Placement.  Workgroups are dispatched to the eight XCDs round-robin by
// workgroup id, so rank r of group p is given id 8 NS (p / 8) + p % 8 + 8 r:
// all ranks land on XCD p % 8 and share its L2.  On a shared L2 a post is:
// plain stores of the data, s_waitcnt vmcnt(0) (the stores have reached L2,
// the L1 being write-through), a workgroup barrier, then a device-scope store
// of the flag; the wait is: a device-scope poll of the peers' flags, a
// barrier, then device-scope loads of the peers' data (ld_xchg: they skip
// this CU's L1 and read the shared L2).  Plain loads would not do: measured on
// the MI355X, a plain load keeps returning a line that another CU of the same
// XCD has since overwritten, also after the workgroup-scope invalidate
// (buffer_inv sc0); the agent-scope invalidate (buffer_inv sc1) makes them
// correct but drops L2 contents the chain kernels still use, which doubled
// their time.  At kernel start the ranks swap their hardware XCC ids with
// device-scope accesses; if they differ (another dispatch order), every post
// and wait of that group also uses the agent-scope release / acquire fences,
// which write back and invalidate the L2 for the other XCD.
//
// Every wait is bounded (by default kTimeoutTicks of the 100 MHz real-time
// counter; the host passes the limit with the launch; a limit of zero makes
// every wait give up before it reads a flag).  A
// rank whose wait expires sets the status word, poisons its own flag so that
// the others stop waiting too, and skips all later waits, so the grid always
// drains; the results of that launch are then undefined and the status word
// reports it.  The kernels are launched cooperatively, so all ranks of a group
// are resident at the same time.
//
// Sync words (uint32, one 256-byte line each, zeroed by the kernel that runs
// before the chain kernel on the same stream), for NG groups:
//   line 0                        status (0 ok, 1 a wait expired)
//   line 1 + NS p + r             flag of rank r of group p (last posted sequence number)
//   line 1 + NS NG + NS p + r     hardware XCC id + 1 of rank r of group p
#pragma once

#include <hip/hip_runtime.h>

namespace e2ttt {

constexpr int kSyncLine = 64;                       // uint32 words per line
constexpr long long kTimeoutTicks = 200000000LL;    // 2 s of the 100 MHz counter
constexpr unsigned kPoison = 0xFFFFFFFFu;

__host__ __device__ constexpr long sync_words(long ngroups, int ns) {
  return kSyncLine * (1 + 2L * ns * ngroups);
}

__device__ __forceinline__ unsigned ld_dev(const unsigned* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_dev(unsigned* p, unsigned v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ int hw_xcc_id() {
  int v;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
  return v & 0xf;
}

// Group index and rank of workgroup b in a launch of NS NG workgroups.
template <int NS>
__device__ __forceinline__ void group_of_block(int b, long& p, int& rank) {
  rank = (b >> 3) % NS;
  p = (long)(b / (8 * NS)) * 8 + (b & 7);
}

// Exchange-slot index of group p among ngroups (a multiple of 8): the groups
// that share an XCD (p mod 8) get consecutive slot blocks, so that each XCD's
// slots form one contiguous range spread over all sets of its L2.  Indexed by
// p itself, the blocks of one XCD's groups would lie 8 blocks (a power-of-two
// multiple of the set span) apart, all on the same L2 sets, and evict each
// other between a post and the peer's read.
__device__ __forceinline__ long slots_of_group(long p, long ngroups) {
  return (p & 7) * (ngroups >> 3) + (p >> 3);
}

// The k-th rank other than `rank`, in increasing order (k < NS - 1).
__device__ __forceinline__ int other_rank(int k, int rank) { return k < rank ? k : k + 1; }

// Sum of the NS partials of one value in rank order: `own` is this rank's,
// peer[k] that of other_rank(k, rank).  Every array index is a compile-time
// constant (the rank only selects), so the partials stay in registers.
template <int NS>
__device__ __forceinline__ float sum_ranks(float own, const float (&peer)[NS - 1], int rank) {
  float acc = 0.0f;
#pragma unroll
  for (int r = 0; r < NS; ++r) {
    const float below = peer[r > 0 ? r - 1 : 0];       // rank r when r > rank
    const float above = peer[r < NS - 1 ? r : 0];      // rank r when r < rank
    const float v = (r == rank) ? own : ((r < rank) ? above : below);
    acc = (r == 0) ? v : acc + v;
  }
  return acc;
}

template <int NS> struct PairX;

// One workgroup per unit: nothing to exchange.
template <> struct PairX<1> {
  int rank = 0;
  long p = 0;
  long xs = 0;
  __device__ void init(unsigned*, long, int*, long long) { p = blockIdx.x; }
  __device__ void post() {}
  __device__ void wait_for(unsigned, int*) {}
  __device__ unsigned seq_now() const { return 0; }
};

template <int NS> struct PairX {
  static_assert(NS >= 2 && NS <= 8, "two to eight workgroups per unit");
  int rank = 0;
  long p = 0;
  long xs = 0;   // the group's exchange-slot index (slots_of_group)
  unsigned* mine = nullptr;
  const unsigned* peer[NS - 1] = {};
  unsigned* status = nullptr;
  unsigned seq = 0;
  bool same_xcc = true;
  bool dead = false;
  long long limit = kTimeoutTicks;

  // s_word: two ints of LDS for broadcasting thread 0's findings; limit: the
  // bound of every wait, in ticks of the 100 MHz real-time counter
  __device__ void init(unsigned* sync, long ngroups, int* s_word, long long limit_ticks) {
    group_of_block<NS>(blockIdx.x, p, rank);
    xs = slots_of_group(p, ngroups);
    limit = limit_ticks;
    status = sync;
    mine = sync + kSyncLine * (1 + NS * p + rank);
#pragma unroll
    for (int k = 0; k < NS - 1; ++k)
      peer[k] = sync + kSyncLine * (1 + NS * p + other_rank(k, rank));
    if (threadIdx.x == 0) {
      unsigned* xm = sync + kSyncLine * (1 + NS * ngroups + NS * p + rank);
      const unsigned id = (unsigned)hw_xcc_id() + 1u;
      st_dev(xm, id);
      const long long t0 = __builtin_amdgcn_s_memrealtime();
      int same = 1, alive = 1;
#pragma unroll
      for (int k = 0; k < NS - 1; ++k) {
        const unsigned* xp = sync + kSyncLine * (1 + NS * ngroups + NS * p + other_rank(k, rank));
        unsigned o = 0;
        // a limit of zero gives up at once, whatever the peer has written (a
        // host-forced expiry); otherwise the flag is read first
        if (limit > 0) {
          while ((o = ld_dev(xp)) == 0u) {
            if (__builtin_amdgcn_s_memrealtime() - t0 > limit) break;
          }
        }
        if (o != id) same = 0;
        if (o == 0u) alive = 0;
      }
      s_word[0] = same;
      s_word[1] = alive;
      if (!alive) { st_dev(status, 1u); st_dev(mine, kPoison); }
    }
    __syncthreads();
    same_xcc = s_word[0] != 0;
    dead = s_word[1] == 0;
    __syncthreads();
  }

  // Publish everything this workgroup stored before the call.  All threads call.
  __device__ void post() {
    // vmcnt(0) through the builtin (encoding 0x0F70: vmcnt 0, expcnt and
    // lgkmcnt unconstrained), which the compiler's own wait tracking sees: an
    // inline-asm wait leaves it believing that loads issued before the post
    // are still in flight, and the first use of one then waits for every
    // memory operation issued after the post as well.  The empty asm keeps
    // the compiler from moving stores below the wait.
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_waitcnt(0x0F70);
    __syncthreads();
    ++seq;
    if (threadIdx.x == 0 && !dead) {
      if (!same_xcc) __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");
      st_dev(mine, seq);
    }
  }

  __device__ unsigned seq_now() const { return seq; }

  // Wait until every other rank has posted at least `target`.  All threads
  // call; the caller has passed a workgroup barrier since the previous call.
  // The call is always a workgroup barrier (also once the group is dead).
  __device__ void wait_for(unsigned target, int* s_word) {
    const bool was_dead = dead;   // uniform over the workgroup
    if (threadIdx.x == 0 && !was_dead) {
      const long long t0 = __builtin_amdgcn_s_memrealtime();
      int ok = 1;
#pragma unroll
      for (int k = 0; k < NS - 1; ++k) {
        if (ok && limit <= 0) ok = 0;   // zero limit: give up at once, as at init
        if (ok) {
          unsigned f;
          while ((f = ld_dev(peer[k])) < target) {
            if (__builtin_amdgcn_s_memrealtime() - t0 > limit) { ok = 0; break; }
          }
          if (f == kPoison) ok = 0;
        }
      }
      if (!ok) { st_dev(status, 1u); st_dev(mine, kPoison); }
      s_word[0] = ok;
    }
    __syncthreads();
    if (was_dead) return;
    if (s_word[0] == 0) dead = true;
    if (!same_xcc) __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent");
  }
};

// Loads of data that another workgroup of the launch has written (exchange
// slots, norm partials): buffer loads with the device-scope bit (sc1), which
// never hit a stale line in this CU's L1, one instruction of up to 16 bytes.
// `buf` is the exchange buffer (the kernel argument: one scalar descriptor
// for every slot; 0x00020000 is the descriptor's fourth word for raw buffer
// access on this GPU family), `base` the wave's slot in it (its byte offset
// goes into the instruction's scalar offset) and `off` the lane's element
// offset from `base`.  Offsets stay far below 2 GiB (the buffers hold a few
// C x d partials per workgroup).
template <class T>
__device__ __forceinline__ T ld_xchg(const void* buf, const T* base, int off) {
  static_assert(sizeof(T) == 4 || sizeof(T) == 8 || sizeof(T) == 16, "4, 8 or 16 bytes");
  const __amdgpu_buffer_rsrc_t r =
      __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(buf), 0, 0x7fffffff, 0x00020000);
  constexpr int kSc1 = 16;   // cache-policy operand: the device-scope bit
  const int sbyte = (int)(reinterpret_cast<const char*>(base) - static_cast<const char*>(buf));
  const int vbyte = off * (int)sizeof(T);
  if constexpr (sizeof(T) == 4) {
    return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b32(r, vbyte, sbyte, kSc1));
  } else if constexpr (sizeof(T) == 8) {
    return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b64(r, vbyte, sbyte, kSc1));
  } else {
    return __builtin_bit_cast(T, __builtin_amdgcn_raw_buffer_load_b128(r, vbyte, sbyte, kSc1));
  }
}
// EPL consecutive floats of an exchange row at element offset `off` from the
// slot `base` in `buf` (16-byte aligned when EPL is a multiple of 4).
template <int EPL>
__device__ __forceinline__ void load_row_xchg(float (&dst)[EPL], const void* buf,
                                              const float* base, int off) {
  if constexpr (EPL % 4 == 0) {
#pragma unroll
    for (int k = 0; k < EPL / 4; ++k) {
      const float4 v = ld_xchg(buf, reinterpret_cast<const float4*>(base), off / 4 + k);
      dst[4 * k] = v.x; dst[4 * k + 1] = v.y; dst[4 * k + 2] = v.z; dst[4 * k + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int q = 0; q < EPL; ++q) dst[q] = ld_xchg(buf, base, off + q);
  }
}



// Sum, in rank order from rank 0 (so every rank forms the same sum), of the
// NS ranks' exchange rows: EPL consecutive floats at element offset `off` of
// each rank's slot, slot(r) giving rank r's.  The loads go out a batch of
// ranks at a time (up to 32 floats in flight per lane) before any is added:
// a row added as soon as it arrives would wait for each load in turn, and each
// such wait also covers every memory operation issued before it.
template <int NS, int EPL, class SLOT>
__device__ __forceinline__ void sum_rows_xchg(float (&acc)[EPL], const void* buf, SLOT slot,
                                              int off) {
  constexpr int RB = (32 / EPL < 1) ? 1 : ((32 / EPL > NS) ? NS : 32 / EPL);
#pragma unroll
  for (int r0 = 0; r0 < NS; r0 += RB) {
    float pr[RB][EPL];
#pragma unroll
    for (int k = 0; k < RB; ++k)
      if (r0 + k < NS) load_row_xchg<EPL>(pr[k], buf, slot(r0 + k), off);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int k = 0; k < RB; ++k)
      if (r0 + k < NS) {
#pragma unroll
        for (int q = 0; q < EPL; ++q) acc[q] = (r0 + k == 0) ? pr[k][q] : acc[q] + pr[k][q];
      }
  }
}
}  // namespace e2ttt
