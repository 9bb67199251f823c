// Steps 1 and 4-5 in one pass: the render of Eq. (1)-(2) and, for the
// fragments whose Id is still missing, the chunk level of their hash (Id of
// Alg. 2), from the same loads.
//
// Hashing is VALU-bound (672 VALU ops per 64-byte block) and the render is
// HBM-bound; done separately they read every byte twice. Here one wave takes
// one (slot, tensor, stripe) task: a stripe is 64 consecutive BLAKE3 chunks of
// the tensor (64 KiB) and lane k owns chunk k, 1 KiB of consecutive bytes,
// i.e. whole rows of the tensor (a row is 64 B .. 1 KiB). Step k loads blocks
// 2k and 2k + 1 of every lane's chunk (128 bytes per lane, a whole cache line,
// lanes 1 KiB apart), one step ahead of their use; the lane compresses them
// into its chunk's chaining value and the pair is written to the lane's rows of
// the merged cache: V and offset-0 K unchanged, other K rotated by R(off) in
// fp64. A half-split pair (j, j + d/2) has its halves half a row apart: in a
// 128-byte row both are in one step, in a 256-byte row the first-half step is
// kept in registers until its partner arrives, in longer rows it is re-read
// from the cache one step before it is needed. The angles depend only on the
// slot and the column, so every lane of a step uses the same (cos, sin) pairs,
// read from the slot's table as wave-uniform values. The output goes through
// the LDS so that each store instruction writes whole 128-byte lines of eight
// chunks; each lane follows its own rows into the merged cache (a chunk may
// cross the end of a head). HBM traffic is the algorithmic minimum (each byte
// read once, written once); the kernel is bound by the VALU work of the hash
// plus the fp64 rotation.
#include <type_traits>

#include "blake3_quad.h"
#include "chunk_ops.h"
#include "fused_geometry.h"
#include "rotate.h"

namespace cm {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
// Persistent grid of up to CUs x CM_FUSED_BLOCKS_PER_CU blocks (fewer when the
// set has fewer tasks); the register budget is capped so that
// CM_FUSED_WAVES_PER_EU waves fit on each SIMD (2 waves: 256 VGPRs, enough for
// three pairs of blocks, the hash state and the fp64 rotation without spills).
// Many more blocks than fit keep the end of the launch short: a block that
// starts late has few tasks.
#ifndef CM_FUSED_BLOCKS_PER_CU
#define CM_FUSED_BLOCKS_PER_CU 32
#endif
#ifndef CM_FUSED_WAVES_PER_EU
#define CM_FUSED_WAVES_PER_EU 2
#endif
#define CM_FUSED_OCCUPANCY __attribute__((amdgpu_waves_per_eu(CM_FUSED_WAVES_PER_EU)))

template <int V>
using IC = std::integral_constant<int, V>;

// Loads are ordinary (cached) accesses: a lane reads a whole 128-byte line
// over two consecutive instructions of the same step, which the caches merge
// (a nontemporal hint would make each 16-byte piece a transfer of its own).
// Stores through the LDS staging write eight whole lines per instruction and
// carry the nontemporal hint (the merged cache is not read back here: measured
// 1.4% faster than cached stores); a lane's own 16-byte pieces (the last stripe
// of a tensor) are stored as ordinary accesses.
__device__ __forceinline__ void load_block(u32x4 (&x)[4], const uint8_t* p) {
#pragma unroll
  for (int q = 0; q < 4; ++q) x[q] = *global_ptr<u32x4>(p + 16 * q);
}

__device__ __forceinline__ void store16(uint8_t* p, u32x4 v) { *(CM_GLOBAL u32x4*)p = v; }

__device__ __forceinline__ void compress_block(B3Cv& st, const u32x4 (&x)[4], uint64_t chunk,
                                               uint32_t flags) {
  uint32_t w[16];
#pragma unroll
  for (int q = 0; q < 4; ++q)
#pragma unroll
    for (int k = 0; k < 4; ++k) w[4 * q + k] = x[q][k];
  b3_compress(st, w, chunk, 64, flags);
}

// N consecutive (cos, sin) pairs j0 .. j0 + N - 1 of a slot's pair-ordered
// table (entry j = cos, sin of off * theta_j). j0 is the same on every lane,
// so the pairs are read by scalar loads (through the constant address space:
// the table is not written while the kernel runs) into scalar registers, which
// the fp64 multiply and FMA take as operands. The table address is made opaque
// first, so that the loads stay where they are used (loop-invariant loads of
// every angle of the slot hoisted out of the step loop would not fit the
// scalar registers).
#define CM_CONST __attribute__((address_space(4)))
template <int N>
__device__ __forceinline__ void pair_angles(const double* __restrict__ table, int j0, double* cs,
                                            double* sn) {
  const double* a = table;
  asm volatile("" : "+s"(a));
  const CM_CONST double* ang = (const CM_CONST double*)a;
#pragma unroll
  for (int e = 0; e < N; ++e) {
    cs[e] = ang[2 * (j0 + e)];
    sn[e] = ang[2 * (j0 + e) + 1];
  }
}

// A wave's LDS staging area: lane l's pair of blocks (eight 16-byte pieces)
// at byte l * 144 + q * 16. The 16 bytes of padding per lane put the pieces q
// of any eight consecutive lanes, and the eight pieces of one lane (read by
// eight consecutive lanes), on distinct LDS banks; each side addresses them
// from one register plus immediate offsets.
constexpr int kStageLane = 144;
constexpr int kStageBytes = 64 * kStageLane;

// Where a task's lanes read and write. A task's address state gives s(b), the
// address of block b of the lane's chunk; d(pos), that of block pos of the
// lane's current output row (nullptr: the row is not written); next_row().
//
// Dense: fragment tensors are contiguous [H][T][row] and the merged cache is
// [2L][H][T_out][row]; a lane's chunk is 1 KiB of consecutive bytes and it
// walks its rows into the merged cache.
template <int RB>
struct DenseTask {
  static constexpr bool kSkips = false;
  const uint8_t* src;     // the lane's chunk
  uint8_t* dst;           // the lane's current row in the merged cache
  int64_t left, T, gap;
  __device__ __forceinline__ const uint8_t* s(int b) const { return src + b * 64; }
  // block b of the chunk dl lanes away (the same stripe)
  __device__ __forceinline__ const uint8_t* s_lane(int b, int dl) const {
    return src + ((int64_t)dl << 10) + b * 64;
  }
  __device__ __forceinline__ uint8_t* d(int pos) const { return dst + pos * 64; }
  __device__ __forceinline__ void next_row() { fused_next_row(dst, left, T, gap, RB); }
};

// QP: stripes of at most 16 chunks are hashed by quads of lanes (the variant
// for sets whose tensors are all shorter than one stripe).
template <bool QP>
struct DenseAddr {
  const int64_t* table;   // per fragment: a row of `stride` int64, tensor pointers from entry 1
  int64_t stride;
  uint8_t* out;
  static constexpr bool kQuadPartial = QP;
  template <int RB>
  __device__ __forceinline__ DenseTask<RB> task(int64_t i, int64_t t, int64_t sidx, int64_t off,
                                                int64_t T, int64_t T_out, int32_t H,
                                                int64_t bytes, int lane, int) const {
    constexpr int RB_SHIFT = __builtin_ctz(RB);
    const FusedLane fl = fused_lane(bytes, sidx, lane, RB_SHIFT, T, T_out, off);
    DenseTask<RB> a;
    a.src = reinterpret_cast<const uint8_t*>(table[i * stride + 1 + t]) + fl.src;
    a.dst = out + t * (int64_t)H * T_out * RB + fl.dst;
    a.left = fl.left;
    a.T = T;
    a.gap = (T_out - T) << RB_SHIFT;   // end of a head's rows -> next head
    return a;
  }
};

// Paged: fragments and the merged cache on pages of a pool (fused_geometry.h).
// At the start of a task each lane resolves the RPC rows of its chunk, where
// each is read and where it goes, into its column of the wave's LDS table
// (entry j * 64 + lane: source row j; (RPC + j) * 64 + lane: destination).
template <int RB>
struct PagedTask {
  static constexpr bool kSkips = true;
  static constexpr int RPC = 1024 / RB;
  static constexpr int BPR = RB / 64;
  static constexpr int RB_SHIFT = __builtin_ctz(RB);
  uint8_t* slice;          // the tensor's (layer, K/V) slice of the pool
  const uint32_t* rows;    // the lane's column of the wave's table
  int j;                   // the lane's current output row (the same on every lane)
  __device__ __forceinline__ const uint8_t* s(int b) const {
    return slice + ((uint64_t)rows[(b / BPR) * 64] << RB_SHIFT) + (b % BPR) * 64;
  }
  __device__ __forceinline__ uint8_t* d(int pos) const {
    const uint32_t r = rows[(RPC + j) * 64];
    return r == kPagedSkipRow ? nullptr : slice + ((uint64_t)r << RB_SHIFT) + pos * 64;
  }
  __device__ __forceinline__ void next_row() { ++j; }
};

struct PagedAddr {
  uint8_t* pool;
  int64_t P;                 // pages
  int32_t b_shift;           // log2 of the rows per page
  const int64_t* table;      // per fragment {T, first}: its page ids start at blocks[first]
  const int32_t* blocks;
  const int32_t* k_table;    // merged block -> page, K and V
  const int32_t* v_table;
  uint32_t* lds;             // the block's tables: [waves][2 * RPC][64]
  static constexpr bool kQuadPartial = false;
  template <int RB>
  __device__ __forceinline__ PagedTask<RB> task(int64_t i, int64_t t, int64_t sidx, int64_t off,
                                                int64_t T, int64_t, int32_t H, int64_t,
                                                int lane, int wave) const {
    constexpr int RPC = PagedTask<RB>::RPC;
    constexpr int RB_SHIFT = PagedTask<RB>::RB_SHIFT;
    PagedTask<RB> a;
    a.slice = pool + ((t * P * H) << (b_shift + RB_SHIFT));
    uint32_t* col = lds + (int64_t)wave * (2 * RPC * 64) + lane;
    a.rows = col;
    a.j = 0;
    const int64_t first = table[2 * i + 1];
    const int32_t* tab = (t & 1) ? v_table : k_table;
    const int64_t q0 = (sidx * 64 + lane) * RPC;   // the chunk's first row in the tensor
    const int64_t rows = (int64_t)H * T;
    ChunkRow c = fused_chunk_row(sidx, lane, RB_SHIFT, T);
#pragma unroll
    for (int r = 0; r < RPC; ++r) {
      uint32_t sr = 0, dr = kPagedSkipRow;
      if (q0 + r < rows) paged_row_pair(blocks, first, tab, P, H, b_shift, off, c, &sr, &dr);
      col[r * 64] = sr;
      col[(RPC + r) * 64] = dr;
      fused_chunk_next(c, T);
    }
    return a;
  }
};

// The chaining values of a stripe of at most 16 chunks of a dense tensor, by
// quads of lanes: lanes 4Q .. 4Q + 3 hash chunk Q (b3_chunk_quad), a chain of
// about half the latency of one lane's. On a small set such stripes are all the
// work and few waves run. stripe: the stripe's first byte; blocks: the tensor's
// 64-byte blocks; cvs: the stripe's first chaining value. Out of line: inlined,
// it makes the 256-byte-row kernel spill.
__device__ __attribute__((noinline)) void quad_hash_stripe(const uint8_t* stripe, int64_t blocks,
                                                           int64_t sidx, bool root, uint8_t* cvs,
                                                           int lane) {
  const int Q = lane >> 2;
  const int64_t left = blocks - (sidx * kStripeChunks + Q) * 16;
  const int nb = left <= 0 ? 0 : (left > 16 ? 16 : (int)left);
  if (nb == 0) return;                                 // uniform over the quad
  const uint8_t* c = stripe + ((int64_t)Q << 10);
  uint32_t lo, hi;
  b3_chunk_quad(lo, hi, nb, (uint64_t)(sidx * kStripeChunks + Q), root, (lane & 1) != 0,
                (lane & 2) != 0,
                [&](int64_t b, uint32_t (&w)[16]) { load_block64(c + b * 64, w); });
  uint32_t* o = reinterpret_cast<uint32_t*>(cvs + (int64_t)Q * 32);
  o[lane & 3] = lo;
  o[4 + (lane & 3)] = hi;
}

// ESIZE: element bytes; STYLE: pairing; RB: row bytes (64 .. 1024); Addr: the
// storage of the fragments and of the merged cache.
template <int ESIZE, int STYLE, int RB, class Addr>
__device__ __forceinline__ void render_hash_body(
    const Addr& addr, int32_t n, const int64_t* __restrict__ plan,
    const int64_t* __restrict__ task_base, const double* __restrict__ angles, int32_t H,
    int32_t d, const uint8_t* __restrict__ select, const int64_t* __restrict__ base0,
    uint8_t* __restrict__ nodes) {
  constexpr int EP = 16 / ESIZE;              // elements per 16-byte piece
  constexpr int BPR = RB / 64;                // blocks per row: 1 .. 16
  constexpr int HBK = BPR / 2;                // blocks per half row (0: a row is one block)
  constexpr int PPR = BPR >= 2 ? BPR / 2 : 1; // steps (pairs of blocks) per row
  constexpr int HP = BPR >= 4 ? BPR / 4 : 0;  // steps per half row when halves span steps
  constexpr bool HALF = STYLE == CM_ROPE_HALF;
  // a half-split pair whose halves are in different steps: the first-half pair
  // of blocks is kept in registers for rows of 256 bytes (one step back) and
  // re-read from the cache for longer rows
  constexpr bool KEEP = HP == 1;
  // the wave index is the same on every lane: say so, so that everything derived
  // from the task (slot, lengths, offsets, step positions, branches) stays in
  // scalar registers
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int64_t waves = (int64_t)gridDim.x * kWaves;
  // Per wave, a staging area through which a pair of blocks of every lane's
  // chunk is handed to the eight lanes that store that chunk's 128 bytes, and
  // the merged-cache address of each lane's two blocks. Lane l stores piece
  // l % 8 of chunk 8 j + l / 8 (j = 0 .. 7).
  __shared__ __attribute__((aligned(16))) uint8_t stage_lds[kWaves][kStageBytes];
  __shared__ uint8_t* dst_lds[kWaves][2][64];
  uint8_t* stage_w = stage_lds[wave] + lane * kStageLane;              // this lane's pieces
  uint8_t* stage_r = stage_lds[wave] + (lane >> 3) * kStageLane + (lane & 7) * 16;
  uint8_t** dst_w = &dst_lds[wave][0][lane];
  uint8_t** dst_r = &dst_lds[wave][(lane & 7) >> 2][lane >> 3];
  const int pq = lane & 3;                         // piece of its block this lane stores
  // the plan and the task bases are read on the device: a plan the host has not
  // seen is rendered as it stands (its length T_out fits the output by contract)
  const int n_u = (int)plan[CM_PLAN_NUNIQUE];
  const int64_t T_out = plan[CM_PLAN_TOUT];
  const int64_t total_tasks = task_base[n];      // 0 for a plan whose status is an error
  for (int64_t task = (int64_t)blockIdx.x * kWaves + wave; task < total_tasks; task += waves) {
    const int s = fused_slot(task_base, n_u, task);
    const int64_t i = plan[CM_PLAN_HEADER + s];
    const int64_t off = plan[CM_PLAN_HEADER + n + s];
    const int64_t T = plan[CM_PLAN_HEADER + 2 * (int64_t)n + s];
    const bool hashing = select[i] == 0;
    const int64_t bytes = (int64_t)H * T * RB;
    const int64_t stripes = stripes_of(bytes);
    const int64_t local = task - task_base[s];
    const int64_t t = local / stripes;             // tensor: 2l + kv
    const int64_t sidx = local - t * stripes;
    const bool rotate = (t & 1) == 0 && off != 0;
    const double* ang = angles + (int64_t)s * d;
    const int64_t m = chunks_of(bytes);
    const int64_t in_stripe = (bytes >> 6) - sidx * kStripeBlocks;
    const bool full = in_stripe >= kStripeBlocks;
    // a last stripe of at most 16 chunks is hashed by quads of lanes in the
    // kernel variant for sets of short tensors (kept out of the other variants:
    // the extra code changes their registers and costs the full-stripe loop)
    constexpr bool kQuadPartial = Addr::kQuadPartial;
    const bool quad_hash = kQuadPartial && hashing && !full && in_stripe <= 16 * 16;
    const uint64_t chunk = (uint64_t)sidx * kStripeChunks + lane;
    const int64_t blocks_left = (bytes >> 6) - (int64_t)chunk * 16;
    const int nb = blocks_left < 0 ? 0 : (blocks_left > 16 ? 16 : (int)blocks_left);
    auto A = addr.template task<RB>(i, t, sidx, off, T, T_out, H, bytes, lane, wave);
    constexpr bool SKIPS = decltype(A)::kSkips;   // rows that are not written
    B3Cv st;
    b3_init(st);
    const uint32_t root = m == 1 ? kB3Root : 0u;
    auto flags = [&](int b, int last) {
      return (b == 0 ? kB3ChunkStart : 0u) | (b == last ? (kB3ChunkEnd | root) : 0u);
    };

    // Rotation in place of block x, block bi of its row (pos of its first
    // piece: bi * 64 bytes), for the pairings a block holds by itself: both
    // halves of a 64-byte row, or interleaved pairs.
    auto rotate_own = [&](u32x4 (&x)[4], int bi) {
      if constexpr (HALF) {
        // the row is this one block: pieces 0, 1 pair with pieces 2, 3
#pragma unroll
        for (int q = 0; q < 2; ++q) {
          double cs[EP], sn[EP];
          pair_angles<EP>(ang, q * EP, cs, sn);
          rotate_pair_half<ESIZE>(x[q], x[q + 2], cs, sn);
        }
      } else {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          double cs[EP / 2], sn[EP / 2];
          pair_angles<EP / 2>(ang, (bi * 64 + 16 * q) / ESIZE / 2, cs, sn);
          x[q] = rotate_piece_il<ESIZE>(x[q], cs, sn);
        }
      }
    };
    // Rotation in place of first-half block a (block bi of its row) and its
    // second-half partner b.
    auto rotate_halves = [&](u32x4 (&a)[4], u32x4 (&b)[4], int bi) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        double cs[EP], sn[EP];
        pair_angles<EP>(ang, bi * (4 * EP) + q * EP, cs, sn);
        rotate_pair_half<ESIZE>(a[q], b[q], cs, sn);
      }
    };
    // Two blocks of every lane (x0 to d0, x1 to d1) through the LDS, so that
    // each store instruction writes eight runs of 128 contiguous bytes.
    auto put2 = [&](const u32x4 (&x0)[4], const u32x4 (&x1)[4], uint8_t* d0, uint8_t* d1) {
      dst_w[0] = d0;
      dst_w[64] = d1;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        *reinterpret_cast<u32x4*>(stage_w + q * 16) = x0[q];
        *reinterpret_cast<u32x4*>(stage_w + 64 + q * 16) = x1[q];
      }
      __builtin_amdgcn_wave_barrier();   // the wave's LDS writes come before its reads
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        uint8_t* p = dst_r[8 * j];
        const u32x4 v = *reinterpret_cast<const u32x4*>(stage_r + j * 8 * kStageLane);
        if constexpr (SKIPS) {
          if (p != nullptr) st_stream(p + pq * 16, v);
        } else {
          st_stream(p + pq * 16, v);
        }
      }
      __builtin_amdgcn_wave_barrier();   // and before the next put's writes
    };

    // Output of step k (blocks 2k, 2k + 1 of every lane's chunk, in y; yp:
    // with half-split pairs spanning steps, the step half a row earlier, the
    // first halves of y's pairs): rotated in place if ROTC, stored, then the
    // lanes move on to the next row after a row's last step. A first-half step
    // of such a row is output with its partner.
    auto emit = [&](auto rotc, int k, u32x4 (&y0)[4], u32x4 (&y1)[4], u32x4 (&yp0)[4],
                    u32x4 (&yp1)[4]) {
      constexpr bool ROT = decltype(rotc)::value;
      const int pp = k % PPR;                     // step of the row
      if constexpr (BPR == 1) {
        // two rows of one block
        if (ROT) { rotate_own(y0, 0); rotate_own(y1, 0); }
        uint8_t* d0 = A.d(0);
        A.next_row();
        put2(y0, y1, d0, A.d(0));
        A.next_row();
        return;
      } else if constexpr (BPR == 2) {
        // one row: halves in y0, y1
        if (ROT) {
          if (HALF) rotate_halves(y0, y1, 0);
          else { rotate_own(y0, 0); rotate_own(y1, 1); }
        }
        put2(y0, y1, A.d(0), A.d(1));
        A.next_row();
        return;
      } else {
        if (ROT && HALF) {
          if (pp < HP) return;                    // output with its partner
          const int pb = 2 * (pp - HP);           // row block of yp0
          rotate_halves(yp0, y0, pb);
          rotate_halves(yp1, y1, pb + 1);
          put2(yp0, yp1, A.d(pb), A.d(pb + 1));
        } else if (ROT) {
          rotate_own(y0, 2 * pp);
          rotate_own(y1, 2 * pp + 1);
        }
        put2(y0, y1, A.d(2 * pp), A.d(2 * pp + 1));
        if (pp == PPR - 1) A.next_row();
      }
    };

    // The steps of a full stripe (every lane owns 16 blocks): step k waits for
    // blocks 2k, 2k + 1 (x, loaded one step earlier); outputs step k - 1 (prev);
    // loads step k + 1 into nx (the last step loads 128 bytes of the slot's
    // angle table instead, lines that stay cached, so that every step issues
    // the same loads), and, when re-reading, the partner pair of
    // step k into pn; then compresses its two blocks. The phases are kept apart
    // so that the fp64 rotation and the compression never hold registers at the
    // same time; every memory operation older than a step's wait was issued a
    // step earlier.
    auto full_stripe = [&](auto hashc, auto rotc) {
      constexpr bool HASH = decltype(hashc)::value;
      constexpr bool ROT = decltype(rotc)::value;
      constexpr bool SPLIT = ROT && HALF && HP > 0;      // halves in different steps
      u32x4 xa0[4], xa1[4], xb0[4], xb1[4], k0[4], k1[4];
      auto load2 = [&](u32x4 (&y0)[4], u32x4 (&y1)[4], int b) {
        if constexpr (SKIPS && BPR == 1) {
          // two rows, each a block
          load_block(y0, A.s(b));
          load_block(y1, A.s(b + 1));
        } else {
          const uint8_t* p = A.s(b);
          load_block(y0, p);
          load_block(y1, p + 64);
        }
      };
      auto step = [&](int k, u32x4 (&x0)[4], u32x4 (&x1)[4], u32x4 (&p0)[4], u32x4 (&p1)[4]) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          launder(x0[q]);
          launder(x1[q]);
        }
        __builtin_amdgcn_sched_barrier(0);
        if (k > 0) {
          // step k - 1 sits in p (the other buffer); its partner in k
          if constexpr (SPLIT && KEEP) {
            if (((k - 1) % PPR) < HP) {
#pragma unroll
              for (int q = 0; q < 4; ++q) {
                k0[q] = p0[q];
                k1[q] = p1[q];
              }
            } else {
              emit(rotc, k - 1, p0, p1, k0, k1);
            }
          } else {
            emit(rotc, k - 1, p0, p1, k0, k1);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        if (k + 1 < 8) {
          load2(p0, p1, (k + 1) * 2);
        } else {
          // the same loads from a line every wave keeps cached: the slot's
          // angle table (at least 128 bytes: d >= 16)
          const uint8_t* hot = reinterpret_cast<const uint8_t*>(ang);
          load_block(p0, hot);
          load_block(p1, hot + 64);
        }
        if constexpr (SPLIT && !KEEP) {
          // the partner pair of step k, needed when step k is output
          if ((k % PPR) >= HP) load2(k0, k1, 2 * (k - HP));
        }
        if constexpr (HASH) {
          compress_block(st, x0, chunk, flags(2 * k, kB3ChunkBlocks - 1));
          compress_block(st, x1, chunk, flags(2 * k + 1, kB3ChunkBlocks - 1));
        }
        __builtin_amdgcn_sched_barrier(0);
      };
      load2(xa0, xa1, 0);
#pragma nounroll
      for (int k = 0; k < 8; k += 2) {
        step(k, xa0, xa1, xb0, xb1);
        step(k + 1, xb0, xb1, xa0, xa1);
      }
      emit(rotc, 7, xb0, xb1, k0, k1);              // step 7's output
    };

    // The last stripe of a tensor (a lane may own fewer than 16 blocks, or
    // none): a block at a time, its partner re-read when it is needed, each lane
    // storing its own blocks; at most one stripe per tensor, so it is kept
    // short in registers.
    auto partial = [&](auto rotc) {
      constexpr bool ROT = decltype(rotc)::value;
      u32x4 x[4], par[4];
      for (int b = 0; b < nb; ++b) {
        const int pos = b & (BPR - 1);
        load_block(x, A.s(b));
        if (ROT && HALF && BPR > 1 && pos >= HBK) load_block(par, A.s(b - HBK));
        if (hashing && !quad_hash) compress_block(st, x, chunk, flags(b, nb - 1));
        bool out = true;
        if (ROT) {
          if (HALF && BPR > 1) {
            if (pos >= HBK) rotate_halves(par, x, pos - HBK);
            else out = false;                     // stored with its partner
          } else {
            rotate_own(x, pos);
          }
        }
        if (out && (!SKIPS || A.d(0) != nullptr)) {
          if (ROT && HALF && BPR > 1) {
            uint8_t* dp = A.d(pos - HBK);
#pragma unroll
            for (int q = 0; q < 4; ++q) store16(dp + 16 * q, par[q]);
          }
          uint8_t* dx = A.d(pos);
#pragma unroll
          for (int q = 0; q < 4; ++q) store16(dx + 16 * q, x[q]);
        }
        if (pos == BPR - 1) A.next_row();
      }
    };

    if (!full) {
      if (rotate) partial(std::true_type{});
      else partial(std::false_type{});
      if constexpr (kQuadPartial) {
        if (quad_hash)
          quad_hash_stripe(A.s_lane(0, -lane), bytes >> 6, sidx, m == 1,
                           nodes + (base0[i] + t * m + (int64_t)sidx * kStripeChunks) * 32, lane);
      }
    } else if (hashing) {
      if (rotate) full_stripe(std::true_type{}, std::true_type{});
      else full_stripe(std::true_type{}, std::false_type{});
    } else {
      if (rotate) full_stripe(std::false_type{}, std::true_type{});
      else full_stripe(std::false_type{}, std::false_type{});
    }
    if (hashing && !quad_hash && nb > 0)
      store_cv(nodes + (base0[i] + t * m + (int64_t)chunk) * 32, st);
  }
}

template <int ESIZE, int STYLE, int RB, bool QP = false>
__global__ __launch_bounds__(kThreads) CM_FUSED_OCCUPANCY void render_hash_kernel(
    const int64_t* __restrict__ table, int64_t stride, int32_t n, const int64_t* __restrict__ plan,
    const int64_t* __restrict__ task_base, const double* __restrict__ angles, int32_t H,
    int32_t d, const uint8_t* __restrict__ select, const int64_t* __restrict__ base0,
    uint8_t* __restrict__ nodes, uint8_t* __restrict__ out) {
  render_hash_body<ESIZE, STYLE, RB>(DenseAddr<QP>{table, stride, out}, n, plan, task_base,
                                     angles, H, d, select, base0, nodes);
}

// The pool is read (fragment pages) and written (the merged cache's fresh
// pages) through the same pointer.
template <int ESIZE, int STYLE, int RB>
__global__ __launch_bounds__(kThreads) CM_FUSED_OCCUPANCY void paged_hash_render_kernel(
    uint8_t* pool, int64_t P, int32_t b_shift, const int64_t* __restrict__ table,
    const int32_t* __restrict__ blocks, const int32_t* __restrict__ k_table,
    const int32_t* __restrict__ v_table, int32_t n, const int64_t* __restrict__ plan,
    const int64_t* __restrict__ task_base, const double* __restrict__ angles, int32_t H,
    int32_t d, const uint8_t* __restrict__ select, const int64_t* __restrict__ base0,
    uint8_t* __restrict__ nodes) {
  __shared__ uint32_t rows_lds[kWaves * 2 * (1024 / RB) * 64];
  render_hash_body<ESIZE, STYLE, RB>(
      PagedAddr{pool, P, b_shift, table, blocks, k_table, v_table, rows_lds}, n, plan, task_base,
      angles, H, d, select, base0, nodes);
}

// Calls go(IC<RB>) for the row size of the set.
template <class Go>
__host__ inline void dispatch_row(int64_t row_bytes, Go&& go) {
  switch ((int)row_bytes) {
    case 64: return go(IC<64>{});
    case 128: return go(IC<128>{});
    case 256: return go(IC<256>{});
    case 512: return go(IC<512>{});
    default: return go(IC<1024>{});
  }
}

}  // namespace

hipError_t launch_render_hash(const SetDesc& s, const HashLayout& hlay, const RenderLayout& rlay,
                              const int64_t* plan_dev, double base, int32_t style,
                              const uint8_t* select, uint8_t* digests, void* out, uint8_t* ws,
                              hipStream_t stream, bool tables_ready, bool prep_ready) {
  uint8_t* hws = ws;
  uint8_t* rws = ws + align_up(hlay.bytes, kWsAlign);
  hipError_t e = hipSuccess;
  if (!tables_ready && (e = launch_hash_prep(s, hlay, hws, stream)) != hipSuccess) return e;
  if (!prep_ready && (e = launch_render_prep(s, rlay, plan_dev, s.n, base, style,
                                             (int32_t)kStripeBlocks, select, rws, stream)) !=
                         hipSuccess)
    return e;
  const uint8_t* hsel = rws + rlay.off_hsel;  // 0: slot delivery whose Id is computed here
  {
    const int64_t* base_tab = reinterpret_cast<const int64_t*>(hws + hlay.off_tables);
    const int64_t* tasks = reinterpret_cast<const int64_t*>(rws + rlay.off_tiles);
    const double* angles = reinterpret_cast<const double*>(rws + rlay.off_angles);
    // the task count is known on the device only; the tasks of every delivery
    // (hlay.tasks) bound it. A persistent grid of a few workgroups per CU, or
    // fewer when there are fewer tasks, strides over it.
    const int64_t cap = (int64_t)device_cu_count() * CM_FUSED_BLOCKS_PER_CU;
    const int64_t want = (hlay.tasks + kWaves - 1) / kWaves;
    const dim3 grid((uint32_t)(want < cap ? (want > 0 ? want : 1) : cap));
    ScopedTiming tm(K_RENDER_HASH, stream);
    uint8_t* nodes = hws + hlay.off_buf0;
    uint8_t* o = reinterpret_cast<uint8_t*>(out);
    bool short_tensors = true;
    for (int i = 0; i < s.n && short_tensors; ++i)
      short_tensors = s.T(i) * token_bytes_of(s) < kStripeBlocks * 64;
    auto go = [&](auto rbc) {
      constexpr int RB = decltype(rbc)::value;
      auto launch = [&](auto kern) {
        hipLaunchKernelGGL(kern, grid, dim3(kThreads), 0, stream, s.table_dev, s.stride, s.n,
                           plan_dev, tasks, angles, s.H, s.d, hsel, base_tab, nodes, o);
      };
      auto pick = [&](auto qpc) {
        constexpr bool QP = decltype(qpc)::value;
        if (s.esize == 2) {
          if (style == CM_ROPE_HALF) launch(render_hash_kernel<2, CM_ROPE_HALF, RB, QP>);
          else launch(render_hash_kernel<2, CM_ROPE_INTERLEAVED, RB, QP>);
        } else {
          if (style == CM_ROPE_HALF) launch(render_hash_kernel<4, CM_ROPE_HALF, RB, QP>);
          else launch(render_hash_kernel<4, CM_ROPE_INTERLEAVED, RB, QP>);
        }
      };
      // every tensor shorter than one stripe (rows up to 256 bytes): every task
      // is a tensor's only, partial stripe, hashed by quads of lanes
      if constexpr (RB <= 256) {
        if (short_tensors) {
          pick(std::true_type{});
          return;
        }
      }
      pick(std::false_type{});
    };
    dispatch_row(s.row_bytes, go);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_hash_tree(s, hlay, hsel, 0, digests, hws, stream);
}

hipError_t launch_paged_render_hash(const PagedDesc& p, const HashLayout& hlay,
                                    const RenderLayout& rlay, const int64_t* plan_dev, double base,
                                    int32_t style, const uint8_t* select, const int32_t* k_table,
                                    const int32_t* v_table, uint8_t* digests, uint8_t* ws,
                                    hipStream_t stream) {
  const SetDesc& s = p.s;
  uint8_t* hws = ws;
  uint8_t* rws = ws + align_up(hlay.bytes, kWsAlign);
  hipError_t e = launch_hash_prep(s, hlay, hws, stream);
  if (e != hipSuccess) return e;
  if ((e = launch_render_prep(s, rlay, plan_dev, s.n, base, style, (int32_t)kStripeBlocks, select,
                              rws, stream)) != hipSuccess)
    return e;
  const uint8_t* hsel = rws + rlay.off_hsel;  // 0: slot delivery whose Id is computed here
  {
    const int64_t* base_tab = reinterpret_cast<const int64_t*>(hws + hlay.off_tables);
    const int64_t* tasks = reinterpret_cast<const int64_t*>(rws + rlay.off_tiles);
    const double* angles = reinterpret_cast<const double*>(rws + rlay.off_angles);
    const int64_t cap = (int64_t)device_cu_count() * CM_FUSED_BLOCKS_PER_CU;
    const int64_t want = (hlay.tasks + kWaves - 1) / kWaves;
    const dim3 grid((uint32_t)(want < cap ? (want > 0 ? want : 1) : cap));
    ScopedTiming tm(K_PAGED_HASH_RENDER, stream);
    uint8_t* nodes = hws + hlay.off_buf0;
    uint8_t* pool = static_cast<uint8_t*>(p.pool);
    auto go = [&](auto rbc) {
      constexpr int RB = decltype(rbc)::value;
      auto launch = [&](auto kern) {
        hipLaunchKernelGGL(kern, grid, dim3(kThreads), 0, stream, pool, p.pages, p.b_shift,
                           s.table_dev, p.blocks_dev, k_table, v_table, s.n, plan_dev, tasks,
                           angles, s.H, s.d, hsel, base_tab, nodes);
      };
      if (s.esize == 2) {
        if (style == CM_ROPE_HALF) launch(paged_hash_render_kernel<2, CM_ROPE_HALF, RB>);
        else launch(paged_hash_render_kernel<2, CM_ROPE_INTERLEAVED, RB>);
      } else {
        if (style == CM_ROPE_HALF) launch(paged_hash_render_kernel<4, CM_ROPE_HALF, RB>);
        else launch(paged_hash_render_kernel<4, CM_ROPE_INTERLEAVED, RB>);
      }
    };
    dispatch_row(s.row_bytes, go);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return launch_hash_tree(s, hlay, hsel, 0, digests, hws, stream);
}

}  // namespace cm
