// Persistent tensor-parallel denoise loop for the batch-1 bf16 expert with
// joint attention: one launch of co-resident workgroups runs every solver step, layer and
// sublayer of vla_denoise (Algorithm 1's loop), with no kernel boundary inside.
//
// The 256 workgroups (4 waves each: one wave per SIMD, so a wave may hold up to
// 512 registers of prefetched operands) form 8 teams of 32: a team is the set
// of workgroups running on one XCD (read from the hardware XCC id at start, so
// the grouping does not rely on the dispatch order) and its traffic stays in
// that XCD's L2.  Team x owns query heads [x*HT, (x+1)*HT) and MLP columns
// [x*F/8, (x+1)*F/8); it recomputes the K/V head its queries share.  Per layer:
//   Q  team GEMM u -> [q of the team's heads | k | v]          team barrier
//   A  attention over [prefix ; chunk] in key splits           team barrier
//   M  merge the splits -> o_team (each rank 1/8 of a tile)     team barrier
//   O  o_team W_o[:, team cols]^T -> delta0                     grid barrier
//   R  x += alpha * (sum of the 8 teams' delta0); adaRMS -> u   team barrier
//   G  team GEMM u -> act(gate) * up (or act(W1 u)) -> h_team   team barrier
//   D  h_team W_d[:, team cols]^T -> delta1                     grid barrier
//   R  x += alpha * sum delta1; adaRMS of the next sublayer     team barrier
// Every team keeps its own copy of the residual stream x, held in registers by
// the workgroup that owns each row (rank r: rows r and r + 32), so R is local
// to a workgroup.  After the last layer R also runs the head, the Euler update
// and the next step's input embedding.  Weights and cached prefix K/V do not
// depend on the step's activations: a workgroup issues their loads before it
// waits at the barrier that precedes the phase using them.
//
// Memory model: data that one workgroup writes and another reads is stored
// with plain (write-through) stores and read with device-coherent (sc1) buffer
// loads; the residual deltas, which cross XCDs, are also stored with sc1.  No
// L2 write-back or invalidate is needed.  Barriers are relaxed agent-scope
// counters; every wait is bounded, and a timeout sets *err, writes NaN into
// the chunk and makes every workgroup leave.
#include <utility>
#include "device_common.h"

namespace {

typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned u32x2_t __attribute__((ext_vector_type(2)));
typedef __amdgpu_buffer_rsrc_t rsrc_t;

constexpr int NTEAM = 8, TSIZE = 32, NWG = NTEAM * TSIZE;
constexpr int NW = 4, NTHR = 64 * NW;    // waves and threads of a workgroup
constexpr int LDX = 16;                  // loads of exchanged data: device-coherent (sc1)
constexpr int STL = 0;                   // stores of exchanged data: plain (write through to L2)
constexpr int SC1 = 16;                  // device-coherent policy of the cross-team deltas
constexpr int KBA_MAX = 2;               // 32-key blocks per attention split
constexpr int MB = 8;                    // key splits one of a vector's 4 merge threads loads (S <= 32)
constexpr float kLog2e = 1.4426950408889634f;
typedef short v4s_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s_t lds_v4s;

// Buffer resource over [base, base + bytes): loads past the end read zero,
// stores past the end are dropped.
VLA_DEV rsrc_t mkr(const void* base, size_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
// Cache policies of exchanged data.  Stores are plain: the L1 writes through,
// so after a store completes its data is in the writer XCD's L2.  Loads of
// data another workgroup wrote are device-coherent (sc1): they miss the CU's
// L1, which may hold a stale copy from an earlier layer.  (L2-coherent sc0
// loads still hit stale L1 lines here, even after an L1 invalidate.)  The
// residual deltas cross XCDs and are written with sc1 stores.
template <int POL>
VLA_DEV uint4 ld16(rsrc_t r, unsigned off) {
  const u32x4_t v = __builtin_amdgcn_raw_buffer_load_b128(r, (int)off, 0, POL);
  return make_uint4(v.x, v.y, v.z, v.w);
}
VLA_DEV uint4 bld16(rsrc_t r, unsigned voff, unsigned soff, int coherent) {
  const u32x4_t v = coherent ? __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, LDX)
                             : __builtin_amdgcn_raw_buffer_load_b128(r, (int)voff, (int)soff, 0);
  return make_uint4(v.x, v.y, v.z, v.w);
}
template <int POL>
VLA_DEV float2 ld8f(rsrc_t r, unsigned off) {
  const u32x2_t v = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, POL);
  return make_float2(__uint_as_float(v.x), __uint_as_float(v.y));
}
template <int POL>
VLA_DEV void st8(rsrc_t r, unsigned off, unsigned lo, unsigned hi) {
  __builtin_amdgcn_raw_buffer_store_b64(u32x2_t{lo, hi}, r, (int)off, 0, POL);
}
template <int POL>
VLA_DEV void st4(rsrc_t r, unsigned off, unsigned v) { __builtin_amdgcn_raw_buffer_store_b32(v, r, (int)off, 0, POL); }
VLA_DEV void st2(rsrc_t r, unsigned off, unsigned short v) { __builtin_amdgcn_raw_buffer_store_b16(v, r, (int)off, 0, STL); }

// Hardware id of the XCD (accelerator complex die) this wave runs on.
VLA_DEV unsigned xcc_id() {
  unsigned v;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(v));
  return v & 0xfu;
}

// ---------------------------------------------------------------------------
// Barriers, without atomics.  Every workgroup owns flag words holding the
// number of barriers it has arrived at: a team flag, stored at team barriers
// with a plain store (only workgroups of the same XCD read it, from that XCD's
// L2, where the line stays), and a grid flag, stored at grid barriers with
// device-coherent stores that other XCDs can see, into eight copies of the
// grid flags 4 KB apart: team x polls copy x, so each copy's lines have 32
// pollers instead of 256 and the copies sit in different memory channels.
// The flags of a team are one 128-byte line, flag[team * 32 + rank].
// Arriving = waiting until this workgroup's stores have completed, then the
// store of the new count.  A team barrier waits until the team's 32 team flags
// reach the count (one load per lane of the first wave), a grid barrier until
// all 256 grid flags of the team's copy do (one 16-byte load per lane).  Flags
// only grow, so a workgroup that is already past the barrier also satisfies it.
struct Sync {
  unsigned* flag;   // 8 copies of [8][32], PERSIST_GFLAG_STRIDE words apart: grid barriers (device-coherent)
  unsigned* tflag;  // [8][32]: team barriers (plain stores: only the team's XCD reads them, from its L2)
  int* err;
  unsigned bk;      // barriers this workgroup has arrived at
  long spin_limit;  // polls before a wait gives up
};

// drain = false: this workgroup stored nothing since its last arrival, so its
// loads in flight need not land first.
template <bool GRID>
VLA_DEV void arrive(Sync& s, int team, int rank, bool drain = true) {
  if (drain) __builtin_amdgcn_s_waitcnt(0);  // this thread's stores have completed
  __syncthreads();
  ++s.bk;
  if (GRID) {
    if (threadIdx.x < NTEAM)   // one copy per thread
      __hip_atomic_store(s.flag + threadIdx.x * PERSIST_GFLAG_STRIDE + team * 32 + rank, s.bk, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  } else if (threadIdx.x == 0) {
    __builtin_amdgcn_raw_buffer_store_b32(s.bk, mkr(s.tflag, (size_t)NWG * 4), (team * 32 + rank) * 4, 0, 0);
  }
}

// Smallest flag this lane of the first wave watches (team: lane < 32 reads
// its teammate's flag; grid: four flags per lane); other threads return ~0.
template <bool GRID>
VLA_DEV unsigned flag_peek(const Sync& s, int team) {
  const int t = threadIdx.x;
  if (t >= 64) return 0xffffffffu;
  if (GRID) {
    // one 16-byte device-coherent load per lane: the 256 flags in one
    // instruction (a quarter of the requests of four 4-byte loads)
    const u32x4_t v =
        __builtin_amdgcn_raw_buffer_load_b128(mkr(s.flag + team * PERSIST_GFLAG_STRIDE, (size_t)NWG * 4), t * 16, 0, LDX);
    return min(min(v.x, v.y), min(v.z, v.w));
  }
  return t < TSIZE ? __hip_atomic_load(s.tflag + team * 32 + t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) : 0xffffffffu;
}

// Returns false (in every thread) if the run must stop.
template <bool GRID>
VLA_DEV bool wait_flags(Sync& s, int team, int* lds_flag, unsigned peek) {
  if (threadIdx.x < 64) {
    const unsigned target = s.bk;
    bool ok = true;
    if (!__all(peek >= target)) {
      long it = 0;
      while (true) {
        // Grid polls about 256 clocks apart: fewer polls on the flag lines in
        // far memory let the flag stores through sooner.  Team polls read the
        // XCD's L2 and go back to back.
        if (GRID) __builtin_amdgcn_s_sleep(4);
        if (__all(flag_peek<GRID>(s, team) >= target)) break;
        if (++it > s.spin_limit) {
          if (threadIdx.x == 0) __hip_atomic_fetch_or(s.err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          ok = false;
          break;
        }
        if ((it & 255) == 0 && __hip_atomic_load(s.err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
          ok = false;
          break;
        }
      }
    }
    if (threadIdx.x == 0) *lds_flag = ok ? 1 : 0;
  }
  __syncthreads();
  return *lds_flag != 0;
}

// ---------------------------------------------------------------------------
// Team GEMM tile: rows [0, M) (M <= 64, four 16-row subtiles), NS 16-row W
// tiles, K <= 1024 in chunks of 128; wave w takes chunks w and w + 4.  Lane
// (r16, g4) holds k = 128 c + 32 v + 8 g4 .. + 8 of row r16 (chunk c), for X
// and W alike.  Operands come through buffer loads whose lane offset is one
// register plus an immediate and whose row-block offset is uniform; X is a
// buffer of exactly M rows of length K, so rows past M read zero.
constexpr int VPL = 4;
constexpr int CPW = 2;

template <int NS>
struct WTile {
  uint4 w[CPW][NS][VPL];
};

// W: [rows][ldw] bf16 (rsrc over the matrix), columns kofs + k; wrow[s] < 0: tile s absent.
template <int NS>
VLA_DEV void prefetch_w(WTile<NS>& t, rsrc_t W, int ldw, int kofs, int K, const int (&wrow)[NS]) {
  // the wave index in a scalar register: the row-block offsets derived from it
  // are scalar, so each load is one instruction (no loop over lane values)
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r16 = lane & 15, g4 = lane >> 4;
#pragma unroll
  for (int j = 0; j < CPW; ++j) {
    const int kc = 128 * (wave + NW * j);
    const unsigned vb = (unsigned)(r16 * ldw + kofs + kc + 8 * g4) * 2u;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      const bool on = kc < K && wrow[s] >= 0;
      const unsigned sb = on ? (unsigned)wrow[s] * (unsigned)ldw * 2u : 0u;
#pragma unroll
      for (int v = 0; v < VPL; ++v) t.w[j][s][v] = on ? bld16(W, vb + 64u * v, sb, 0) : make_uint4(0, 0, 0, 0);
    }
  }
}

// acc[ms][s] over this wave's chunks.  X is an exchanged activation in the
// tiled layout [K/32][M][32] bf16 (so one load instruction of a wave reads 16
// rows x 64 contiguous bytes = 1 KB); rows past M read zero.
VLA_DEV unsigned xtile_off(int m, int k, int M) { return (unsigned)(((k >> 5) * M + m) * 64 + (k & 31) * 2); }

// The X operand is staged through LDS: the wave copies its NCH x VPL groups
// of 4 blocks of 1 KB (16 rows x 32 k) with direct-to-LDS buffer loads, all in
// flight at once and holding no registers, into its own XSTAGE-byte slice;
// lane l of a block lands at byte 16 l, which is the 16 bytes lane l feeds to
// the MFMA.  Each (j, v) group is read back after its own loads have landed
// (in-order vmcnt), so the MFMAs of early groups overlap the later loads.
// Lanes of absent rows and chunks past K get offsets past the buffer, and an
// out-of-range direct-to-LDS load writes zeros, so those operands are zero
// (the weights of chunks past K are zero too).  Every acc[ms][s] sums its
// k-products in the order (j, v), as a register-staged form would.
constexpr int XSTAGE = CPW * VPL * 4 * 1024;   // LDS bytes per wave

// Buffer descriptor words of [base, base + bytes) in SGPRs (the layout
// mkr builds: stride 0, bounds-checked, zero past the end).
VLA_DEV u32x4_t rsrc_words(const void* base, unsigned bytes) {
  const unsigned long long p = (unsigned long long)(uintptr_t)base;
  return u32x4_t{(unsigned)__builtin_amdgcn_readfirstlane((unsigned)p),
                 (unsigned)__builtin_amdgcn_readfirstlane((unsigned)(p >> 32)) & 0xffffu,
                 (unsigned)__builtin_amdgcn_readfirstlane(bytes), 0x00020000u};
}
// One wave-wide device-coherent (sc1) buffer load of 16 bytes per lane into
// LDS at base + off + 16 lane (off wave-uniform; the LDS address is taken from
// base, the kernel's LDS array, and offset, so the compiler needs no null check).  Written as asm so that the compiler
// adds no waits of its own for it; the caller's vmcnt waits order it.
VLA_DEV void dma_x16(const u32x4_t& rs, unsigned voff, unsigned soff, unsigned char* base, unsigned off) {
  typedef __attribute__((address_space(3))) unsigned char lds_u8;
  const unsigned lb = __builtin_amdgcn_readfirstlane((unsigned)(uintptr_t)(lds_u8*)base + off);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen sc1 lds"
               : : "s"(lb), "v"(voff), "s"(rs), "s"(soff) : "memory", "m0");
}
// One wave-wide load of 4 bytes per lane into LDS at base + off + 4 lane, with the default cache policy.  Used only to bring lines into
// the XCD's L2 (the LDS copy is never read); asm, like dma_x16, and waited for
// by the next full wait.
VLA_DEV void touch_l2(const u32x4_t& rs, unsigned voff, unsigned char* base, unsigned off) {
  typedef __attribute__((address_space(3))) unsigned char lds_u8;
  const unsigned lb = __builtin_amdgcn_readfirstlane((unsigned)(uintptr_t)(lds_u8*)base + off);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dword %1, %2, 0 offen lds" : : "s"(lb), "v"(voff), "s"(rs) : "memory", "m0");
}
// As dma_x16, with the default cache policy (read-only data).
VLA_DEV void dma_x16_ro(const u32x4_t& rs, unsigned voff, unsigned soff, unsigned char* base, unsigned off) {
  typedef __attribute__((address_space(3))) unsigned char lds_u8;
  const unsigned lb = __builtin_amdgcn_readfirstlane((unsigned)(uintptr_t)(lds_u8*)base + off);
  asm volatile("s_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, %3 offen lds"
               : : "s"(lb), "v"(voff), "s"(rs), "s"(soff) : "memory", "m0");
}
template <int N>
VLA_DEV void vm_wait_mem() { asm volatile("s_waitcnt vmcnt(%0)" : : "n"(N) : "memory"); }

// NCH: the wave's K chunks (K <= 128 NW NCH); FOLD (M <= 50): the fourth
// 16-row subtile holds at most rows 48 and 49, and those rows of all the
// wave's groups come in with one load (lane l: group l / 8, row 48 + (l / 4) % 2,
// k part l % 4) instead of one mostly out-of-range load per group.  A load
// costs the address unit the same whether its lanes are in range or not.
template <int NS, int NCH, bool FOLD>
VLA_DEV void tile_mma(f32x4 (&acc)[4][NS], const WTile<NS>& t, const void* xbase, unsigned xbytes, int K, int M,
                      unsigned char* stage) {
  static_assert(NCH >= 1 && NCH <= CPW && (!FOLD || NCH * VPL <= 8), "tile_mma shape");
  constexpr int NG = NCH * VPL;            // (j, v) groups of the wave
  constexpr int LPG = FOLD ? 3 : 4;        // loads per group
  const int lane = threadIdx.x & 63, wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int r16 = lane & 15, g4 = lane >> 4;
  unsigned char* ws = stage + wave * XSTAGE;
  const u32x4_t rs = rsrc_words(xbase, xbytes);
  // The weight tile (and every other load in flight) must land before the
  // first MFMA anyway.  Waiting here, with a wait the compiler sees, clears
  // its count of outstanding loads, so it adds no vmcnt(0) of its own after
  // the asm loads below, which it cannot count and which would stall every
  // group until the last one has landed.
  __builtin_amdgcn_s_waitcnt(vm_wait(0));
  if constexpr (FOLD) {   // rows 48, 49 of every group, into group 0's fourth block
    const int gg = lane >> 3, rr = 48 + ((lane >> 2) & 1);
    const int kc = 128 * (wave + NW * (gg / VPL));
    const unsigned off = (gg < NG && kc < K && rr < M)
                             ? (unsigned)((((kc >> 5) + gg % VPL) * M + rr) * 64 + (lane & 3) * 16)
                             : 0x7ffffff0u;
    dma_x16(rs, off, 0u, stage, (unsigned)(wave * XSTAGE + 3 * 1024));
  }
  unsigned vo[4];
#pragma unroll
  for (int ms = 0; ms < 4; ++ms) vo[ms] = (16 * ms + r16 < M) ? (unsigned)(r16 * 64 + g4 * 16) : 0x7ffffff0u;
#pragma unroll
  for (int j = 0; j < NCH; ++j) {
    const int kc = 128 * (wave + NW * j);
#pragma unroll
    for (int v = 0; v < VPL; ++v)
#pragma unroll
      for (int ms = 0; ms < LPG; ++ms) {
        const unsigned so = kc < K ? (unsigned)(((kc >> 5) + v) * M * 64 + ms * 16 * 64) : 0x7ffffff0u;
        dma_x16(rs, vo[ms], so, stage, (unsigned)(wave * XSTAGE + ((j * VPL + v) * 4 + ms) * 1024));
      }
  }
#pragma unroll
  for (int ms = 0; ms < 4; ++ms)
#pragma unroll
    for (int s = 0; s < NS; ++s) acc[ms][s] = f32x4{0.f, 0.f, 0.f, 0.f};
  // group g = (j, v): wait until only the later groups' loads are in flight
  // (the folded load is older than all of them)
  auto group = [&]<int G>(std::integral_constant<int, G>) {
    constexpr int j = G / VPL, v = G % VPL;
    vm_wait_mem<LPG * (NG - 1 - G)>();
    uint4 x[4];
#pragma unroll
    for (int ms = 0; ms < LPG; ++ms) x[ms] = *reinterpret_cast<const uint4*>(ws + (G * 4 + ms) * 1024 + lane * 16);
    if constexpr (FOLD) {
      const uint4 f = *reinterpret_cast<const uint4*>(ws + 3 * 1024 + (G * 8 + (r16 & 1) * 4 + g4) * 16);
      x[3] = r16 < 2 ? f : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int ms = 0; ms < 4; ++ms)
#pragma unroll
      for (int s = 0; s < NS; ++s) mma16(acc[ms][s], x[ms], t.w[j][s][v], bf16_t());
  };
  [&]<int... G>(std::integer_sequence<int, G...>) {
    (group(std::integral_constant<int, G>{}), ...);
  }(std::make_integer_sequence<int, NG>{});
}

// Sum the 4 waves' tiles through LDS (red: 4 * 4 * NS * 64 f32x4); afterwards
// wave w holds the full 16-row subtile w in acc[0][s].
template <int NS>
VLA_DEV void tile_reduce(f32x4 (&acc)[4][NS], f32x4* red) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int ms = 0; ms < 4; ++ms)
#pragma unroll
    for (int s = 0; s < NS; ++s) red[((wave * 4 + ms) * NS + s) * 64 + lane] = acc[ms][s];
  __syncthreads();
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    f32x4 r = red[((0 * 4 + wave) * NS + s) * 64 + lane];
#pragma unroll
    for (int w = 1; w < NW; ++w) r += red[((w * 4 + wave) * NS + s) * 64 + lane];
    acc[0][s] = r;
  }
}

// ---------------------------------------------------------------------------
template <int HD>
struct PLds {
  static constexpr int KP = HD + 8;    // K row pitch (bf16)
  // V row-major [32 keys][HD], unpadded: 16-byte chunk c of key k at slot
  // c ^ 2 (k % 4); read as the V^T operand with transposing LDS loads
  static constexpr size_t KBYTES = 32 * KP * 2;
  static constexpr size_t BUF = KBYTES + (size_t)32 * HD * 2;
};

size_t lds_main(int hd) {
  const size_t att = KBA_MAX * (hd == 256 ? PLds<256>::BUF : hd == 128 ? PLds<128>::BUF : PLds<64>::BUF);
  const size_t red2 = (size_t)NW * 4 * 2 * 64 * 16;
  return att > red2 ? att : red2;
}

// FOLD: the chunk has at most 50 rows (see tile_mma).
template <int HD, int DPT, bool FOLD>
__global__ __launch_bounds__(NTHR, 1) void persist_kernel(PersistArgs a) {
  using L = PLds<HD>;
  constexpr int VPR = HD / 8;              // 16-byte vectors per K/V row
  constexpr int NQV = HD / 32;             // Q fragments per lane
  constexpr int DTL = HD / 16;             // dim tiles of O^T
  constexpr int NKI = (KBA_MAX * 32 * VPR + NTHR - 1) / NTHR;  // K items per thread
  constexpr int OKS = 8;                   // O-projection k-steps of 32 (K = HT * hd <= 256)
  constexpr int OTW = 2;                   // O-projection 16-column tiles per rank
  extern __shared__ __align__(16) unsigned char smem[];
  __shared__ int flag;
  __shared__ float red_s[2][NW];
  __shared__ float sa[2][32];              // a of this workgroup's rows (broadcast copy)
  __shared__ float hv[2][NW][32];          // head partial sums per wave
  __shared__ PLayer lt[PERSIST_MAX_LAYERS];

  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r16 = lane & 15, g4 = lane >> 4;
  // Team = the XCD this workgroup runs on, rank = its arrival order there, so
  // the team-local exchange through the XCD's L2 is coherent whatever order
  // the dispatcher used.  A team with more than 32 members (a part or mode
  // without 8 XCDs of 32 CUs) stops the run through the error flag.
  __shared__ int s_team, s_rank;
  if (tid == 0) {
    const unsigned x = xcc_id();
    s_team = (int)(x % NTEAM);
    s_rank = (int)__hip_atomic_fetch_add(a.sync + PERSIST_RANK_OFF + (x % NTEAM), 1u, __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT);
    if (s_rank >= TSIZE || x >= (unsigned)NTEAM)
      __hip_atomic_fetch_or(a.err, 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  if (s_rank >= TSIZE) return;
  const int team = s_team, rank = s_rank;
  const int n = a.n, d = a.d, HT = a.HT, A = a.A;
  const int HTD = HT * HD, QW = (HT + 2) * HD, F8 = a.F / 8, S = a.nsplit;
  const int QT = (n + 15) / 16;
  const int dq = a.H * HD, dkv = a.G * HD;
  const int gteam = (team * HT * a.G) / a.H;        // K/V head of the team's queries
  f32x4* red = reinterpret_cast<f32x4*>(smem);
  for (int i = tid; i < a.L; i += NTHR) lt[i] = a.layers[i];
  const bf16_t* kvbase = reinterpret_cast<const bf16_t*>(a.cp->kv_cache);

  Sync sy{a.sync, a.sync + PERSIST_TFLAG_OFF, a.err, 0u, a.spin_limit};
  unsigned long long* trace = !a.trace ? nullptr
                              : a.trace_all ? a.trace + (size_t)(team * TSIZE + rank) * PERSIST_TRACE_WG
                              : (rank == 0 ? a.trace + (size_t)team * PERSIST_TRACE_MAX : nullptr);
  const int tcap = a.trace_all ? PERSIST_TRACE_WG : PERSIST_TRACE_MAX;
  int tev = 0;
  auto mark = [&]() {
    if (trace && tid == 0 && tev < tcap) trace[tev] = __builtin_amdgcn_s_memrealtime();
    ++tev;
  };
  // A barrier timed out: leave, marking the chunk as failed (NaN).
  auto bail = [&]() {
    for (int i = tid; i < n * a.A; i += NTHR) a.cp->actions_out[i] = __int_as_float(0x7fc00000);
  };

  // team-local workspace
  const rsrc_t Ur = mkr((const bf16_t*)a.u + (size_t)team * n * d, (size_t)n * d * 2);
  const rsrc_t Qr = mkr((const bf16_t*)a.qkv + (size_t)team * n * QW, (size_t)n * QW * 2);
  const rsrc_t APr = mkr((const bf16_t*)a.apart + (size_t)team * S * n * HTD, (size_t)S * n * HTD * 2);
  const rsrc_t ASr = mkr(a.astat + (size_t)team * S * n * HT * 2, (size_t)S * n * HT * 8);
  const rsrc_t Hr = mkr((const bf16_t*)a.hbuf + (size_t)team * n * F8, (size_t)n * F8 * 2);
  const void* ubase = (const bf16_t*)a.u + (size_t)team * n * d;     // the GEMM phases' X operands
  const void* hbase = (const bf16_t*)a.hbuf + (size_t)team * n * F8;
  const rsrc_t OMr = mkr((const bf16_t*)a.omerged + (size_t)team * n * HTD, (size_t)n * HTD * 2);
  const rsrc_t Dr = mkr(a.delta, (size_t)2 * NTEAM * n * d * 4);   // [buf][team][n][d]

  // rows of this workgroup and their residual stream (columns tid*DPT + e)
  const int mrow[2] = {rank, rank + TSIZE};
  const bool mok[2] = {rank < n, rank + TSIZE < n};
  float xr[2][DPT];
  float areg[2] = {0.f, 0.f};              // thread j < A: a[mrow][j]
  for (int r = 0; r < 2; ++r)
    if (mok[r] && tid < A) areg[r] = a.a0[(size_t)mrow[r] * A + tid];

  const size_t modstep = (size_t)a.L * 2 * 3 * d;
  auto gam = [&](int k, int l, int j) { return a.mods + k * modstep + ((size_t)l * 2 + j) * 3 * d; };

  // ---- row-phase pieces ----------------------------------------------------
  // block sums of v0 (row 0) and v1 (row 1)
  auto sum2 = [&](float v0, float v1, float& s0, float& s1) {
    v0 = wave_sum(v0);
    v1 = wave_sum(v1);
    if (lane == 0) {
      red_s[0][wave] = v0;
      red_s[1][wave] = v1;
    }
    __syncthreads();
    s0 = 0.f;
    s1 = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      s0 += red_s[0][w];
      s1 += red_s[1][w];
    }
    __syncthreads();
  };
  // Row-phase loads are branch-free: an absent row gets an offset past the
  // end of its buffer resource (the load returns zero), so every load of a
  // helper is issued before the first wait.
  const int c0 = tid * DPT;                // this thread's residual columns
  constexpr unsigned OOB = 0x7ffffff0u;
  auto ldf = [&](float (&v)[DPT], const float* src) {   // DPT contiguous fp32
    if constexpr (DPT == 4) {
      const float4 t = *reinterpret_cast<const float4*>(src);
      v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
    } else {
      const float2 t = *reinterpret_cast<const float2*>(src);
      v[0] = t.x; v[1] = t.y;
    }
  };
  auto ldbf = [&](float (&v)[DPT], rsrc_t r, unsigned off) {   // DPT contiguous bf16
    if constexpr (DPT == 4) {
      const u32x2_t t = __builtin_amdgcn_raw_buffer_load_b64(r, (int)off, 0, 0);
      v[0] = __uint_as_float(t.x << 16); v[1] = __uint_as_float(t.x & 0xffff0000u);
      v[2] = __uint_as_float(t.y << 16); v[3] = __uint_as_float(t.y & 0xffff0000u);
    } else {
      const unsigned t = __builtin_amdgcn_raw_buffer_load_b32(r, (int)off, 0, 0);
      v[0] = __uint_as_float(t << 16); v[1] = __uint_as_float(t & 0xffff0000u);
    }
  };
  // adaRMS of both rows with (g, b); u (bf16) to the team's U
  auto norm_store = [&](const float* g, const float* b) {
    float gg[DPT], bb[DPT];
    ldf(gg, g + c0);
    ldf(bb, b + c0);
    float ss[2] = {0.f, 0.f};
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int e = 0; e < DPT; ++e) ss[r] += xr[r][e] * xr[r][e];
    float t0, t1;
    sum2(ss[0], ss[1], t0, t1);
    const float rs[2] = {1.0f / sqrtf(t0 / (float)d + a.eps), 1.0f / sqrtf(t1 / (float)d + a.eps)};
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      float u[DPT];
#pragma unroll
      for (int e = 0; e < DPT; ++e) u[e] = xr[r][e] * rs[r] * (1.0f + gg[e]) + bb[e];
      const unsigned off = mok[r] ? xtile_off(mrow[r], c0, n) : OOB;   // tiled [d/32][n][32]
      if constexpr (DPT == 4) st8<STL>(Ur, off, pack_bf16x2(u[0], u[1]), pack_bf16x2(u[2], u[3]));
      else st4<STL>(Ur, off, pack_bf16x2(u[0], u[1]));
    }
  };
  // x += alpha * (sum over teams of delta[buf]), summed in team order
  auto resid = [&](int buf, const float* alpha) {
    float al[DPT];
    ldf(al, alpha + c0);
    float dv[2][NTEAM][DPT];
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int y = 0; y < NTEAM; ++y) {
        const unsigned off = mok[r] ? (unsigned)((((size_t)buf * NTEAM + y) * n + mrow[r]) * d + c0) * 4u : OOB;
        if constexpr (DPT == 4) {
          const uint4 v = ld16<SC1>(Dr, off);
          dv[r][y][0] = __uint_as_float(v.x);
          dv[r][y][1] = __uint_as_float(v.y);
          dv[r][y][2] = __uint_as_float(v.z);
          dv[r][y][3] = __uint_as_float(v.w);
        } else {
          const float2 v = ld8f<SC1>(Dr, off);
          dv[r][y][0] = v.x;
          dv[r][y][1] = v.y;
        }
      }
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int e = 0; e < DPT; ++e) {
        float sum = 0.f;
#pragma unroll
        for (int y = 0; y < NTEAM; ++y) sum += dv[r][y][e];
        xr[r][e] += al[e] * sum;   // absent rows: xr stays 0 (their deltas read as 0)
      }
  };
  // x = a W_in^T + xs + E_pos (input embedding of the chunk tokens).  W_in is
  // the zero-padded [d][32] copy; sa holds a with zeros past A.
  const rsrc_t WIr = mkr(a.w_in, (size_t)d * 32 * 2);
  const rsrc_t EPr = mkr(a.e_pos, (size_t)n * d * 2);
  const rsrc_t WOr = mkr(a.w_out, (size_t)A * d * 2);
  auto embed = [&]() {
    if (tid < 32) {
      sa[0][tid] = tid < A ? areg[0] : 0.f;
      sa[1][tid] = tid < A ? areg[1] : 0.f;
    }
    uint4 wv[DPT][4];
#pragma unroll
    for (int e = 0; e < DPT; ++e)
#pragma unroll
      for (int q = 0; q < 4; ++q) wv[e][q] = ld16<0>(WIr, (unsigned)((c0 + e) * 32 + 8 * q) * 2u);
    float base[DPT], ep[2][DPT];
    ldf(base, a.xs + c0);
#pragma unroll
    for (int r = 0; r < 2; ++r) ldbf(ep[r], EPr, mok[r] ? (unsigned)(mrow[r] * d + c0) * 2u : OOB);
    __syncthreads();
#pragma unroll
    for (int e = 0; e < DPT; ++e) {
      float f[32];
#pragma unroll
      for (int q = 0; q < 4; ++q) unpack16(wv[e][q], f + 8 * q, bf16_t());
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        float v = base[e] + ep[r][e];
#pragma unroll
        for (int t = 0; t < 32; ++t) v += sa[r][t] * f[t];
        xr[r][e] = mok[r] ? v : 0.f;
      }
    }
    __syncthreads();
  };
  // head v = u_f W_out^T + b_out on the final adaRMS (fp32), then the Euler
  // update of a (threads j < A); writes the chunk on the last step.
  auto head = [&](int k) {
    const float* g = a.modf + (size_t)k * 2 * d;
    const float* b = g + d;
    float wo_[32][DPT];                    // W_out[j][c0 ..]; rows j >= A read zero
#pragma unroll
    for (int j = 0; j < 32; ++j) ldbf(wo_[j], WOr, j < A ? (unsigned)(j * d + c0) * 2u : OOB);
    float gg[DPT], bb[DPT];
    ldf(gg, g + c0);
    ldf(bb, b + c0);
    float ss[2] = {0.f, 0.f};
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int e = 0; e < DPT; ++e) ss[r] += xr[r][e] * xr[r][e];
    float t0, t1;
    sum2(ss[0], ss[1], t0, t1);
    const float rs[2] = {1.0f / sqrtf(t0 / (float)d + a.eps), 1.0f / sqrtf(t1 / (float)d + a.eps)};
    float uf[2][DPT];
#pragma unroll
    for (int e = 0; e < DPT; ++e)
#pragma unroll
      for (int r = 0; r < 2; ++r) uf[r][e] = xr[r][e] * rs[r] * (1.0f + gg[e]) + bb[e];
#pragma unroll
    for (int j = 0; j < 32; ++j) {
      float p0 = 0.f, p1 = 0.f;
#pragma unroll
      for (int e = 0; e < DPT; ++e) {
        p0 += uf[0][e] * wo_[j][e];
        p1 += uf[1][e] * wo_[j][e];
      }
      p0 = wave_sum(p0);
      p1 = wave_sum(p1);
      if (lane == 0) {
        hv[0][wave][j] = p0;
        hv[1][wave][j] = p1;
      }
    }
    __syncthreads();
    const CallParams* cp = a.cp;
    const float dt = cp->tau[k + 1] - cp->tau[k];
    if (tid < A) {
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        float v = a.b_out[tid];
#pragma unroll
        for (int w = 0; w < NW; ++w) v += hv[r][w][tid];
        areg[r] += dt * v;
      }
      if (k == a.T - 1 && team == 0) {
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          if (!mok[r]) continue;
          float o = areg[r];
          if (cp->act_std) o *= cp->act_std[tid];
          if (cp->act_mean) o += cp->act_mean[tid];
          cp->actions_out[(size_t)mrow[r] * A + tid] = o;
        }
      }
    }
    __syncthreads();
  };

  // ---- phase pieces ----------------------------------------------------------
  const int NTQ = QW / 16;                 // QKV tiles of the team
  auto qkv_rows = [&](int (&wrow)[2], int (&ocol)[2]) {
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      const int t = rank + TSIZE * s;
      wrow[s] = -1;
      ocol[s] = -1;
      if (t >= NTQ) continue;
      const int c = 16 * t;                // local column
      if (c < HTD) wrow[s] = team * HTD + c;
      else if (c < HTD + HD) wrow[s] = dq + gteam * HD + (c - HTD);
      else wrow[s] = dq + dkv + gteam * HD + (c - HTD - HD);
      ocol[s] = c;
    }
  };
  const int npairs = F8 / 16;              // 16-column groups of h per team (one per rank)
  auto gu_rows = [&](int (&wrow)[2]) {
    const int p = rank;
    if (p >= npairs) {
      wrow[0] = wrow[1] = -1;
    } else if (a.glu) {
      wrow[0] = team * 2 * F8 + 32 * p;
      wrow[1] = wrow[0] + 16;
    } else {
      wrow[0] = team * F8 + 16 * p;
      wrow[1] = -1;
    }
  };
  const int DCOL = d / TSIZE;             // down-projection columns per rank (16 or 32)
  auto dn_rows = [&](int (&wrow)[2]) {
    wrow[0] = rank * DCOL;
    wrow[1] = DCOL > 16 ? rank * DCOL + 16 : -1;
  };

  // attention split of this rank
  const int npre = a.P, nself = n;
  const int nbp = (npre + 31) / 32;
  // Key splits: the prefix blocks in groups of kba, then one split per block
  // of chunk-token keys (whose K / V arrive with this step's Q phase, so the
  // split that holds them is the phase's longest path).
  const int nps = (nbp + a.kba - 1) / a.kba;
  const bool att_on = rank < S;
  const bool pre_split = __builtin_amdgcn_readfirstlane(rank < nps ? 1 : 0) != 0;   // holds prefix keys
  const int jbeg = rank < nps ? rank * a.kba : nbp + (rank - nps);
  const int nblk = att_on ? (rank < nps ? min(nbp, jbeg + a.kba) : jbeg + 1) - jbeg : 0;
  uint4 kpre[NKI], vpre[NKI];
  auto prefetch_kv = [&](int l) {
    const bf16_t* kc = kvbase + lt[l].cache_off + (size_t)gteam * npre * HD;
    const bf16_t* vc = kc + (size_t)a.G * npre * HD;
    const rsrc_t KR = mkr(kc, (size_t)npre * HD * 2), VR = mkr(vc, (size_t)npre * HD * 2);
#pragma unroll
    for (int q = 0; q < NKI; ++q) {
      const int i = tid + q * NTHR;
      const int jb = i / (32 * VPR), rr = i - jb * 32 * VPR;
      const int kr = rr / VPR, cv = rr - kr * VPR;
      const int j = jbeg + jb, key = j * 32 + kr;
      const bool ok = i < nblk * 32 * VPR && j < nbp;   // keys past the prefix read zero
      kpre[q] = ld16<0>(KR, ok ? (unsigned)(key * HD + cv * 8) * 2u : OOB);
      vpre[q] = ld16<0>(VR, ok ? (unsigned)(key * HD + cv * 8) * 2u : OOB);
    }
  };

  // LDS staging of one attention split's blocks: item i is 16-byte vector
  // i % VPR of key row (i / VPR) % 32 of block i / (32 VPR), for K and V alike.
  // K rows go to their padded rows, V rows to their swizzled slots.
  auto put_kv = [&](int i, uint4 k, uint4 v) {
    const int jb = i / (32 * VPR), rr = i - jb * 32 * VPR;
    const int kr = rr / VPR, cv = rr - kr * VPR;
    bf16_t* kl = reinterpret_cast<bf16_t*>(smem + jb * L::BUF);
    *reinterpret_cast<uint4*>(kl + kr * L::KP + cv * 8) = k;
    unsigned char* vl = smem + jb * L::BUF + L::KBYTES;
    *reinterpret_cast<uint4*>(vl + kr * HD * 2 + (cv ^ (2 * (kr & 3))) * 16) = v;
  };
  // Prefix K / V of the split, from the prefetched registers (chunk blocks get
  // zeros here and their keys after the barrier).
  auto stage_prefix = [&]() {
#pragma unroll
    for (int q = 0; q < NKI; ++q) {
      const int i = tid + q * NTHR;
      if (i < nblk * 32 * VPR) put_kv(i, kpre[q], vpre[q]);
    }
  };

  WTile<2> wq, wg, wd;
  const int CW = d / TSIZE;                // O-projection columns per rank (16 or 32)
  const int ot = rank / 8, ocb = rank % 8; // merge: query tile and column eighth of this rank
  // The rank's W_o rows (OTW tiles of 16) over K = HT * hd, loaded once per
  // workgroup by direct-to-LDS loads (every wave of the O phase uses the same
  // operand) into the LDS past the O phase's activation tile: block
  // (t, ks) of 1 KB holds the 16 bytes lane l feeds to the MFMA at byte 16 l.
  // Absent blocks read zero.  Nothing in the merge phase uses that LDS, and
  // the merge's arrival waits for these loads.
  constexpr int WOFF = 64 * (256 + 8) * 2;   // past the largest activation tile
  auto prefetch_wo = [&](int l) {
    const u32x4_t rs = rsrc_words(lt[l].wo, (unsigned)((size_t)d * dq * 2));
    const unsigned vb = (unsigned)(r16 * dq + team * HTD + 8 * g4) * 2u;
#pragma unroll
    for (int i = 0; i < OTW * OKS / NW; ++i) {
      const int b = wave + NW * i, t = b / OKS, ks = b - t * OKS;
      const bool on = 16 * t < CW && 32 * ks < HTD;
      const unsigned so = on ? (unsigned)(rank * CW + 16 * t) * (unsigned)dq * 2u : 0x7ffffff0u;
      dma_x16_ro(rs, vb + 64u * ks, so, smem, (unsigned)(WOFF + b * 1024));
    }
  };

  __syncthreads();
  mark();
  {
    int wr[2], oc[2];
    qkv_rows(wr, oc);
    prefetch_w<2>(wq, mkr(lt[0].wqkv, (size_t)(dq + 2 * dkv) * d * 2), d, 0, d, wr);
  }
  embed();
  norm_store(gam(0, 0, 0), gam(0, 0, 0) + d);
  mark();
  arrive<false>(sy, team, rank);
      if (!wait_flags<false>(sy, team, &flag, flag_peek<false>(sy, team))) return bail();
  mark();

  for (int k = 0; k < a.T; ++k) {
    for (int l = 0; l < a.L; ++l) {
      const PLayer& ly = lt[l];
      // ---- Q: u -> [q | k | v] of the team -----------------------------------
      {
        int wr[2], oc[2];
        qkv_rows(wr, oc);
        f32x4 acc[4][2];
        tile_mma<2, DPT / 2, FOLD>(acc, wq, ubase, (unsigned)(n * d * 2), d, n, smem);
        __syncthreads();
        tile_reduce<2>(acc, red);
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          if (oc[s] < 0) continue;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int m = 16 * wave + 4 * g4 + i;
            if (m < n) st2(Qr, (unsigned)(m * QW + oc[s] + r16) * 2u, f2bf(acc[0][s][i]));
          }
        }
      }
      mark();
      arrive<false>(sy, team, rank);
      const unsigned pk1 = flag_peek<false>(sy, team);
      // Prefix K / V of a prefix split, independent of this step: loaded and
      // staged while the team arrives.  Other ranks load nothing here (a
      // chunk split's block is filled after the barrier).
      if (pre_split) {
        prefetch_kv(l);
        stage_prefix();
      }
      if (!wait_flags<false>(sy, team, &flag, pk1)) return bail();
      mark();

      // ---- A: attention partials of key split `rank` ---------------------------
      if (att_on) {
        // Q fragments of wave (hh, qs) and this step's k, v of the chunk tokens
        // that fall in the split's blocks: all issued at once, branch-free
        // (prefix blocks and rows past the chunk read zero).
        const int hh = wave / QT, qs = wave - hh * QT;
        const bool qwave = hh < HT;
        const int qrow = 16 * qs + r16;
        uint4 qf[NQV];
        const unsigned qb = (unsigned)(qrow * QW + hh * HD + g4 * (HD / 4)) * 2u;
#pragma unroll
        for (int c = 0; c < NQV; ++c) qf[c] = ld16<LDX>(Qr, qwave ? qb + 16u * c : OOB);
        // A split holding chunk-token keys holds one block of them (jbeg >=
        // nbp): one block's items per thread (every wave-wide load costs the
        // address unit about as much whether its lanes are in range or not).
        constexpr int NKC = 32 * VPR / NTHR;
        const bool chunk = jbeg >= nbp;
        uint4 kch[NKC], vch[NKC];
#pragma unroll
        for (int q = 0; q < NKC; ++q) {
          const int i = tid + q * NTHR;
          const int kr = i / VPR, cv = i - kr * VPR;
          const int key = (jbeg - nbp) * 32 + kr;
          const bool ok = chunk && key < nself;
          const unsigned off = ok ? (unsigned)(key * QW + HTD + cv * 8) * 2u : OOB;
          kch[q] = ld16<LDX>(Qr, off);
          vch[q] = ld16<LDX>(Qr, ok ? off + HD * 2u : OOB);
        }
        if (chunk) {
#pragma unroll
          for (int q = 0; q < NKC; ++q) put_kv(tid + q * NTHR, kch[q], vch[q]);
        }
        __syncthreads();
        if (qwave) {
          f32x4 o[DTL];
#pragma unroll
          for (int dd = 0; dd < DTL; ++dd) o[dd] = f32x4{0.f, 0.f, 0.f, 0.f};
          // A split holds at most KBA_MAX blocks: every score of the split is
          // computed first and kept in registers, so the exact maximum is
          // known before any exponent and the accumulators never need a
          // rescale.  Score tile t of block jb, row rho: key
          // 32 jb + 8 (rho / 4) + 4 t + rho % 4; the lane holds keys
          // 32 jb + 8 g4 + 4 t + i of query r16.
          const float sc = a.scale * kLog2e;
          f32x4 sv[KBA_MAX][2];
          float mrun = -INFINITY;
#pragma unroll
          for (int jb = 0; jb < KBA_MAX; ++jb) {
            const int j = jbeg + jb;
            const int cnt = jb >= nblk ? 0 : j < nbp ? min(32, npre - j * 32) : min(32, nself - (j - nbp) * 32);
            const bf16_t* kl = reinterpret_cast<const bf16_t*>(smem + jb * L::BUF);
#pragma unroll
            for (int t = 0; t < 2; ++t) {
              sv[jb][t] = f32x4{0.f, 0.f, 0.f, 0.f};
              if (jb < nblk) {
                const int kr = 8 * (r16 >> 2) + 4 * t + (r16 & 3);
                const bf16_t* krow = kl + kr * L::KP + g4 * (HD / 4);
                // every operand of the tile is read before its first MFMA, so
                // the LDS latencies overlap
                uint4 kf[NQV];
#pragma unroll
                for (int c = 0; c < NQV; ++c) kf[c] = *reinterpret_cast<const uint4*>(krow + c * 8);
                __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                for (int c = 0; c < NQV; ++c) mma16(sv[jb][t], kf[c], qf[c], bf16_t());
              }
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                const int kr = 8 * g4 + 4 * t + i;
                sv[jb][t][i] = (kr < cnt) ? sv[jb][t][i] * sc : -INFINITY;
                mrun = fmaxf(mrun, sv[jb][t][i]);
              }
            }
          }
          mrun = fmaxf(mrun, __shfl_xor(mrun, 16, 64));
          mrun = fmaxf(mrun, __shfl_xor(mrun, 32, 64));
          float lrun = 0.0f;
#pragma unroll
          for (int jb = 0; jb < KBA_MAX; ++jb) {
            if (jb >= nblk) continue;
            const bf16_t* vl = reinterpret_cast<const bf16_t*>(smem + jb * L::BUF + L::KBYTES);
            float p[8];
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
              for (int i = 0; i < 4; ++i) {
                p[4 * t + i] = exp2f(sv[jb][t][i] - mrun);
                lrun += p[4 * t + i];
              }
            uint4 pb;
            pb.x = pack_bf16x2(p[0], p[1]);
            pb.y = pack_bf16x2(p[2], p[3]);
            pb.z = pack_bf16x2(p[4], p[5]);
            pb.w = pack_bf16x2(p[6], p[7]);
            // A operand of dim tile dd: V^T rows 16 dd + r16, keys 8 g4 .. + 7,
            // from two transposing reads.  Within 16 lanes, lane i receives
            // element i % 4 of the 8-byte blocks that lanes i/4, i/4 + 4,
            // i/4 + 8 and i/4 + 12 address; lane p addresses key row
            // 8 g4 + p / 4 (+ 4 for the second read) at dims 16 dd + 4 (p % 4)
            // and so gets 4 consecutive keys of dim 16 dd + p.
            constexpr int VG = DTL < 4 ? DTL : 4;   // V^T operands read ahead of their MFMAs
            const unsigned char* vb = reinterpret_cast<const unsigned char*>(vl) + (8 * g4 + (r16 >> 2)) * HD * 2 + (r16 & 1) * 8;
#pragma unroll
            for (int d0 = 0; d0 < DTL; d0 += VG) {
              uint4 va[VG];
#pragma unroll
              for (int i = 0; i < VG; ++i) {
                const int dd = d0 + i;
                const unsigned char* ap = vb + ((2 * dd + ((r16 & 3) >> 1)) ^ (2 * (r16 >> 2))) * 16;
                const v4s_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(ap));
                const v4s_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(ap + 4 * HD * 2));
                va[i] = make_uint4(((uint32_t)(uint16_t)lo[0]) | ((uint32_t)(uint16_t)lo[1] << 16),
                                   ((uint32_t)(uint16_t)lo[2]) | ((uint32_t)(uint16_t)lo[3] << 16),
                                   ((uint32_t)(uint16_t)hi[0]) | ((uint32_t)(uint16_t)hi[1] << 16),
                                   ((uint32_t)(uint16_t)hi[2]) | ((uint32_t)(uint16_t)hi[3] << 16));
              }
#pragma unroll
              for (int i = 0; i < VG; ++i) mma16(o[d0 + i], va[i], pb, bf16_t());
            }
          }
          lrun += __shfl_xor(lrun, 16, 64);
          lrun += __shfl_xor(lrun, 32, 64);
          // lane holds O^T[dim 16 dd + 4 g4 + i][query r16]
          if (qrow < n) {
            const float inv = lrun > 0.0f ? 1.0f / lrun : 0.0f;
            const unsigned rowoff = (unsigned)((rank * n + qrow) * HTD + hh * HD);
#pragma unroll
            for (int dd = 0; dd < DTL; ++dd)
              st8<STL>(APr, (rowoff + 16 * dd + 4 * g4) * 2u, pack_bf16x2(o[dd][0] * inv, o[dd][1] * inv),
                   pack_bf16x2(o[dd][2] * inv, o[dd][3] * inv));
            if (g4 == 0)
              st8<STL>(ASr, (unsigned)(((rank * n + qrow) * HT + hh) * 2) * 4u, __float_as_uint(mrun),
                   __float_as_uint(lrun));
          }
        }
      } else if (S < TSIZE) {
        // A rank without a key split brings its share of the team's MLP
        // weights of this layer into the XCD's L2 (one 4-byte load per 64
        // bytes): the gate / up rows, then the down projection's block.  The
        // G and D phases' weight loads, issued at the barriers before them,
        // then hit there instead of waiting for HBM, and the polls queued
        // behind those loads return sooner.  Started about 1 us into the
        // phase, after the key splits' own loads; not waited for (see below).
        const int nwv = (TSIZE - S) * NW, w0 = (rank - S) * NW + wave;
        const size_t gurows = (size_t)(a.glu ? 2 : 1) * F8;
        const unsigned gub = (unsigned)(gurows * d * 2);
        const u32x4_t rg = rsrc_words((const bf16_t*)ly.wgu + (size_t)team * gurows * d, gub);
        const unsigned db = (unsigned)((size_t)d * F8 * 2);
        const u32x4_t rd = rsrc_words((const bf16_t*)ly.wd + (size_t)team * d * F8, db);
        __builtin_amdgcn_s_sleep(40);
        for (int it = w0; it < (int)(gub / 4096u); it += nwv) touch_l2(rg, (unsigned)it * 4096u + lane * 64u, smem, (unsigned)wave * 256u);
        for (int it = w0; it < (int)(db / 4096u); it += nwv) touch_l2(rd, (unsigned)it * 4096u + lane * 64u, smem, (unsigned)wave * 256u);
      }
      mark();
      // A rank without a key split stored nothing here and arrives at once;
      // its L2 loads land before the merge phase's loads (in-order returns) and
      // before its next full wait, ahead of the O phase's LDS use.
      arrive<false>(sy, team, rank, __builtin_amdgcn_readfirstlane(att_on ? 1 : 0) != 0);
      const unsigned pk2 = flag_peek<false>(sy, team);
      prefetch_wo(l);
      if (!wait_flags<false>(sy, team, &flag, pk2)) return bail();
      mark();

      // ---- M: merge the key splits; rank (t, cb) merges query tile t, columns
      // [cb * HTD / 8, (cb + 1) * HTD / 8) of the team's heads into o_team.  Four
      // threads share each 8-column vector: thread quarter q merges splits
      // q, q+4, ... (one round of loads), then the four combine through lane
      // shuffles.
      // a merge thread loads splits qtr, qtr + 4, ...: MBX = 4 covers up to 16 splits
      auto merge = [&]<int MBX>(std::integral_constant<int, MBX>) {
      if (ot < QT) {
        const int cw8 = HTD / 8;                          // merged columns per rank (8 .. 32)
        const int nv = 16 * (cw8 / 8);                    // 16-byte vectors (<= 64)
        const int i = tid >> 2, qtr = tid & 3;
        if (i < nv) {
          const int rr = i / (cw8 / 8), cv = ocb * (cw8 / 8) + (i - rr * (cw8 / 8));
          const int m = 16 * ot + rr;
          const int hh = (cv * 8) / HD;
          const bool live = m < n;
          float acc8[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) acc8[e] = 0.f;
          float mx = -INFINITY, tot = 0.f;
          uint4 v[MBX];
          float2 st[MBX];
#pragma unroll
          for (int q = 0; q < MBX; ++q) {
            const int sp = qtr + 4 * q;
            const bool ok = live && sp < S;   // absent splits read (0, 0): skipped below
            st[q] = ld8f<LDX>(ASr, ok ? (unsigned)(((sp * n + m) * HT + hh) * 2) * 4u : OOB);
            v[q] = ld16<LDX>(APr, ok ? (unsigned)((sp * n + m) * HTD + cv * 8) * 2u : OOB);
          }
#pragma unroll
          for (int q = 0; q < MBX; ++q) {
            if (st[q].y <= 0.f) continue;
            const float mnew = fmaxf(mx, st[q].x);
            const float corr = exp2f(mx - mnew);
            const float w = st[q].y * exp2f(st[q].x - mnew);
            float f[8];
            unpack16(v[q], f, bf16_t());
#pragma unroll
            for (int e = 0; e < 8; ++e) acc8[e] = acc8[e] * corr + w * f[e];
            tot = tot * corr + w;
            mx = mnew;
          }
#pragma unroll
          for (int sh = 1; sh <= 2; sh <<= 1) {
            const float mo = __shfl_xor(mx, sh, 64), to = __shfl_xor(tot, sh, 64);
            const float mn = fmaxf(mx, mo);
            const float cs = tot > 0.f ? exp2f(mx - mn) : 0.f, co = to > 0.f ? exp2f(mo - mn) : 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) acc8[e] = acc8[e] * cs + __shfl_xor(acc8[e], sh, 64) * co;
            tot = tot * cs + to * co;
            mx = mn;
          }
          if (live && qtr == 0) {
            const float inv = tot > 0.f ? 1.0f / tot : 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) acc8[e] *= inv;
            const uint4 pk = pack16(acc8, bf16_t());
            st8<STL>(OMr, (unsigned)(m * HTD + cv * 8) * 2u, pk.x, pk.y);
            st8<STL>(OMr, (unsigned)(m * HTD + cv * 8 + 4) * 2u, pk.z, pk.w);
          }
        }
      }
      };
      if (S <= 16) merge(std::integral_constant<int, 4>{});
      else merge(std::integral_constant<int, MB>{});
      mark();
      arrive<false>(sy, team, rank);
      if (!wait_flags<false>(sy, team, &flag, flag_peek<false>(sy, team))) return bail();
      mark();

      // ---- O: o_team (all rows) times W_o[rank's CW columns][team heads]^T;
      // wave w takes query tile w --------------------------------------------------
      {
        bf16_t* otile = reinterpret_cast<bf16_t*>(smem);   // [64][HTD + 8]
        const int OP = HTD + 8;
        const int nv = 64 * (HTD / 8);      // <= 8 vectors per thread (HTD <= 256)
        uint4 ov[8];
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int i = tid + q * NTHR;
          const int rr = i / (HTD / 8), cv = i - rr * (HTD / 8);
          ov[q] = ld16<LDX>(OMr, i < nv ? (unsigned)(rr * HTD + cv * 8) * 2u : OOB);   // rows past n read zero
        }
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          const int i = tid + q * NTHR;
          const int rr = i / (HTD / 8), cv = i - rr * (HTD / 8);
          if (i < nv) *reinterpret_cast<uint4*>(otile + rr * OP + cv * 8) = ov[q];
        }
        __syncthreads();
        if (wave < QT) {
#pragma unroll
          for (int t = 0; t < OTW; ++t) {
            const int cl = 16 * t;
            if (cl >= CW) break;
            f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < OKS; ++ks) {
              if (32 * ks >= HTD) break;
              const uint4 av = *reinterpret_cast<const uint4*>(otile + (16 * wave + r16) * OP + 32 * ks + 8 * g4);
              const uint4 wv = *reinterpret_cast<const uint4*>(smem + WOFF + (t * OKS + ks) * 1024 + lane * 16);
              mma16(acc, av, wv, bf16_t());
            }
            const int col = rank * CW + cl + r16;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int m = 16 * wave + 4 * g4 + i;
              if (m < n) st4<SC1>(Dr, (unsigned)((((size_t)0 * NTEAM + team) * n + m) * d + col) * 4u, __float_as_uint(acc[i]));
            }
          }
        }
      }
      mark();
      arrive<true>(sy, team, rank);
      const unsigned pk3 = flag_peek<true>(sy, team);
      {
        int wr[2];
        gu_rows(wr);
        prefetch_w<2>(wg, mkr(ly.wgu, (size_t)(a.glu ? 2 : 1) * a.F * d * 2), d, 0, d, wr);
      }
      if (!wait_flags<true>(sy, team, &flag, pk3)) return bail();
      mark();

      // ---- R: attention residual, adaRMS of the MLP sublayer --------------------
      resid(0, gam(k, l, 0) + 2 * d);
      norm_store(gam(k, l, 1), gam(k, l, 1) + d);
      mark();
      arrive<false>(sy, team, rank);
      if (!wait_flags<false>(sy, team, &flag, flag_peek<false>(sy, team))) return bail();
      mark();

      // ---- G: u -> h of the team's MLP columns ------------------------------------
      {
        f32x4 acc[4][2];
        tile_mma<2, DPT / 2, FOLD>(acc, wg, ubase, (unsigned)(n * d * 2), d, n, smem);
        __syncthreads();
        tile_reduce<2>(acc, red);
        if (rank < npairs) {
          const int f = 16 * rank + r16;
          // one branch on the (uniform) activation for the lane's four values
          float g[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) g[i] = acc[0][0][i];
          switch (a.act) {
            case ACT_SILU:
#pragma unroll
              for (int i = 0; i < 4; ++i) g[i] = silu_f(g[i]);
              break;
            case ACT_GELU:
#pragma unroll
              for (int i = 0; i < 4; ++i) g[i] = gelu_tanh_f(g[i]);
              break;
            case ACT_RELU2:
#pragma unroll
              for (int i = 0; i < 4; ++i) { const float r = fmaxf(g[i], 0.0f); g[i] = r * r; }
              break;
            default: break;
          }
          if (a.glu) {
#pragma unroll
            for (int i = 0; i < 4; ++i) g[i] *= acc[0][1][i];
          }
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int m = 16 * wave + 4 * g4 + i;
            if (m < n) st2(Hr, xtile_off(m, f, n), f2bf(g[i]));   // tiled [F8/32][n][32]
          }
        }
      }
      mark();
      arrive<false>(sy, team, rank);
      const unsigned pk4 = flag_peek<false>(sy, team);
      {
        int wr[2];
        dn_rows(wr);
        prefetch_w<2>(wd, mkr((const bf16_t*)ly.wd + (size_t)team * d * F8, (size_t)d * F8 * 2), F8, 0, F8, wr);
      }
      if (!wait_flags<false>(sy, team, &flag, pk4)) return bail();
      mark();

      // ---- D: h_team W_d[:, team cols]^T -> delta1 -----------------------------------
      {
        int wr[2];
        dn_rows(wr);
        f32x4 acc[4][2];
        tile_mma<2, 1, FOLD>(acc, wd, hbase, (unsigned)(n * F8 * 2), F8, n, smem);   // K = F / 8 <= 512
        __syncthreads();
        tile_reduce<2>(acc, red);
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          if (wr[s] < 0) continue;
          const int col = wr[s] + r16;
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const int m = 16 * wave + 4 * g4 + i;
            if (m < n) st4<SC1>(Dr, (unsigned)((((size_t)1 * NTEAM + team) * n + m) * d + col) * 4u, __float_as_uint(acc[0][s][i]));
          }
        }
      }
      const bool last_layer = l == a.L - 1;
      const bool last = last_layer && k == a.T - 1;
      mark();
      arrive<true>(sy, team, rank);
      const unsigned pk5 = flag_peek<true>(sy, team);
      {
        int wr[2], oc[2];
        qkv_rows(wr, oc);
        const int nl = last_layer ? 0 : l + 1;
        prefetch_w<2>(wq, mkr(lt[nl].wqkv, (size_t)(dq + 2 * dkv) * d * 2), d, 0, d, wr);
      }
      if (!wait_flags<true>(sy, team, &flag, pk5)) return bail();
      mark();

      // ---- R: MLP residual; next sublayer's adaRMS (or head, Euler, embedding) ---
      resid(1, gam(k, l, 1) + 2 * d);
      if (!last_layer) {
        norm_store(gam(k, l + 1, 0), gam(k, l + 1, 0) + d);
      } else {
        head(k);
        if (k + 1 < a.T) {
          embed();
          norm_store(gam(k + 1, 0, 0), gam(k + 1, 0, 0) + d);
        }
      }
      if (!last) {
        mark();
        arrive<false>(sy, team, rank);
      if (!wait_flags<false>(sy, team, &flag, flag_peek<false>(sy, team))) return bail();
        mark();
      }
    }
  }
  mark();
}

}  // namespace

bool persist_supported(int d, int hd, int H, int G, int F, int n, int P, int A, int glu, int* kba, int* nsplit) {
  if (!(d == 512 || d == 1024)) return false;   // R: d / 256 columns per thread; O: d / 8 columns per rank
  if (!(hd == 64 || hd == 128 || hd == 256)) return false;
  if (H % NTEAM != 0 || G < 1 || H % G != 0) return false;
  const int HT = H / NTEAM;
  // all heads of a team share one K/V head
  for (int t = 0; t < NTEAM; ++t)
    if ((t * HT * G) / H != ((t * HT + HT - 1) * G) / H) return false;
  if (HT * hd > 256) return false;           // O-projection K and the attention Q registers
  if (n < 1 || n > 2 * TSIZE) return false;  // two rows per rank, four 16-row subtiles
  const int QT = (n + 15) / 16;
  if (HT * QT > NW) return false;            // attention: one wave per (head, query tile)
  if ((HT + 2) * hd / 16 > 2 * TSIZE) return false;  // QKV tiles: two per rank
  if (F % 128 != 0 || F / 8 > 1024 || F / 128 > TSIZE) return false;  // h groups: one per rank
  (void)glu;
  if (A < 1 || A > 32) return false;         // head and embedding registers
  const int nbp = (P + 31) / 32, nbs = (n + 31) / 32;   // prefix and chunk-token key blocks
  int k = 1;
  while ((nbp + k - 1) / k + nbs > TSIZE) ++k;
  if (k < 2 && nbp > 16) k = 2;              // fewer, larger splits: shorter attention phase
  if (k > KBA_MAX) return false;
  *kba = k;
  *nsplit = (nbp + k - 1) / k + nbs;
  return true;
}

size_t persist_lds_bytes(int hd, int HT) {
  const size_t otile = (size_t)64 * (HT * hd + 8) * 2;
  const size_t mainb = lds_main(hd);
  const size_t xst = (size_t)NW * XSTAGE;   // the GEMM phases' staged activations
  const size_t m2 = mainb > otile ? mainb : otile;
  return m2 > xst ? m2 : xst;
}

namespace {
template <bool FOLD>
const void* persist_fn_t(int hd, int dpt) {
  switch (hd * 10 + dpt) {
    case 2564: return reinterpret_cast<const void*>(&persist_kernel<256, 4, FOLD>);
    case 2562: return reinterpret_cast<const void*>(&persist_kernel<256, 2, FOLD>);
    case 1284: return reinterpret_cast<const void*>(&persist_kernel<128, 4, FOLD>);
    case 1282: return reinterpret_cast<const void*>(&persist_kernel<128, 2, FOLD>);
    case 644: return reinterpret_cast<const void*>(&persist_kernel<64, 4, FOLD>);
    case 642: return reinterpret_cast<const void*>(&persist_kernel<64, 2, FOLD>);
    default: return nullptr;
  }
}
// chunks of at most 50 rows take the folded-tail form of the GEMM phases
const void* persist_fn(int hd, int d, int n) {
  return n <= 50 ? persist_fn_t<true>(hd, d / NTHR) : persist_fn_t<false>(hd, d / NTHR);
}
}  // namespace

bool persist_resident(int d, int hd, int HT) {
  const void* fns[2] = {persist_fn(hd, d, 1), persist_fn(hd, d, 64)};
  if (!fns[0] || !fns[1]) return false;
  int dev = 0, cus = 0, nb = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus != NWG)
    return false;
  const size_t lds = persist_lds_bytes(hd, HT);
  for (const void* fn : fns) {
    if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess) return false;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fn, NTHR, lds) != hipSuccess || nb < 1) return false;
  }
  return true;
}

// A plain launch: the plan builder has checked that every workgroup fits on
// the device at once (persist_resident), and every barrier wait of the kernel
// is bounded, so a workgroup that never started would end the run through the
// error word, not hang it.
hipError_t launch_persist(const PersistArgs& a, hipStream_t s) {
  const size_t lds = persist_lds_bytes(a.hd, a.HT);
  void* args[] = {const_cast<PersistArgs*>(&a)};
  const void* fn = persist_fn(a.hd, a.d, a.n);
  if (!fn) return hipErrorInvalidValue;
  hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  return hipLaunchKernel(fn, dim3(NWG), dim3(NTHR), args, lds, s);
}
