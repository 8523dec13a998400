// Shared device-side building blocks for the attention kernels (gfx950 only).
//
// Every kernel in this library has the same shape.  A workgroup owns a block
// of "stationary" rows (query rows in the row-major kernels, key rows in the
// column-major kernels), held as MFMA B-operands in registers.  It streams
// the other side of the attention matrix through LDS in tiles of kBS = 32
// rows, and per tile it
//   1. forms transposed score-like tiles  T[s][t] = X_s . Y_t   (s streamed,
//      t stationary) with v_mfma_f32_16x16x32_bf16 (or 16x16x4f32), where the
//      streamed row-major tile is the A-operand read straight out of LDS;
//   2. does the elementwise work on those tiles in fp32 registers (the output
//      layout puts the stationary row on lane & 15, so row scalars are
//      per-lane values);
//   3. accumulates Acc^T[dim][t] += X^T[dim][s] . T^T[s][t], with the
//      streamed tile transposed on the fly by ds_read_b64_tr_b16 and the
//      score tile reused in registers as the B-operand.
// Accumulators therefore live transposed: lane l holds dims 16*nb + 4*(l>>4)
// + r (r = 0..3) of stationary row 16*mb + (l & 15).
//
// Lane layouts (checked on gfx950 with an in-bounds probe):
//   16x16x32 bf16 A: lane l -> row l&15, k = 8*(l>>4) + e, e = 0..7
//                 B: lane l -> col l&15, same k;   C: lane l -> rows 4*(l>>4)+r, col l&15
//   16x16x4 f32   A: lane l -> row l&15, k = l>>4;  B: col l&15, k = l>>4; C as above
//   ds_read_b64_tr_b16: in each group of 16 lanes, lane j gives the address of
//   4 consecutive 16-bit elements (row j/4, cols 4*(j%4)..+3 of a 4x16 block);
//   lane i receives column i of that block (4 elements, rows 0..3).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace fb {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short shortx4 __attribute__((ext_vector_type(4)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

#define FB_LDS __attribute__((address_space(3)))

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// forward: growth of a row maximum (log2 units) that forces a rescale
constexpr float kRescaleLog2 = 8.f;
constexpr float kRescaleP = 256.f;   // 2^kRescaleLog2
constexpr int kBS = 32;  // streamed rows per tile (two 16-row MFMA sub-blocks)

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }
__device__ __forceinline__ int wave_id() { return threadIdx.x >> 6; }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Sum / max over the four lanes that share lane & 15 (the four k-groups).
__device__ __forceinline__ float group_sum(float x) {
  x += __shfl_xor(x, 16);
  x += __shfl_xor(x, 32);
  return x;
}
__device__ __forceinline__ float group_max(float x) {
  x = fmaxf(x, __shfl_xor(x, 16));
  x = fmaxf(x, __shfl_xor(x, 32));
  return x;
}

// ---------------------------------------------------------------------------
// Element-type policy.  A "chunk" is the 16 bytes one lane contributes to a
// score MFMA step: 8 bf16 (one 16x16x32 MFMA) or 4 fp32 (four 16x16x4 MFMAs).
// Lane group g = l >> 4 covers dims [kk*kKC + g*kKC/4, +kKC/4) of chunk kk,
// i.e. byte offset 64*kk + 16*g in the row, for both element types.
// ---------------------------------------------------------------------------
template <typename T> struct Elt;

template <> struct Elt<bf16> {
  static constexpr int kKC = 32;
  // score step over one chunk
  static __device__ __forceinline__ floatx4 mma_chunk(u32x4 a, u32x4 b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                   __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
  }
  // A-operand of the accumulate step: 16 dims x 32 streamed rows, transposed
  struct AFrag { bf16x8 v; };
  // B-operand of the accumulate step: this lane's stationary row against the
  // 8 streamed rows {4g+r, 16+4g+r}; slot i = 4*h + r
  struct TFrag {
    bf16x8 v;
    __device__ __forceinline__ void set(int i, float x) { v[i] = (bf16)x; }
  };
  static __device__ __forceinline__ floatx4 mma_acc(const AFrag& a, const TFrag& b, floatx4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a.v, b.v, c, 0, 0, 0);
  }
  // store 4 consecutive output elements (fp32 -> bf16, round to nearest even)
  static __device__ __forceinline__ void store4(bf16* p, floatx4 x) {
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
    bf16x4 y;
    y[0] = (bf16)x[0]; y[1] = (bf16)x[1]; y[2] = (bf16)x[2]; y[3] = (bf16)x[3];
    *(u32x2*)p = __builtin_bit_cast(u32x2, y);
  }
  static __device__ __forceinline__ floatx4 load4(const bf16* p) {
    typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
    bf16x4 y = __builtin_bit_cast(bf16x4, *(const u32x2*)p);
    return floatx4{(float)y[0], (float)y[1], (float)y[2], (float)y[3]};
  }
  // dot product of two chunks (used for D = rowsum(dO * O))
  static __device__ __forceinline__ float dot_chunk(u32x4 a, u32x4 b) {
    bf16x8 x = __builtin_bit_cast(bf16x8, a), y = __builtin_bit_cast(bf16x8, b);
    float s = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) s = __builtin_fmaf((float)x[e], (float)y[e], s);
    return s;
  }
};

template <> struct Elt<float> {
  static constexpr int kKC = 16;
  // The chunk is reinterpreted as a whole floatx4 before taking elements:
  // bit-casting single u32 vector elements inside an unrolled loop made this
  // compiler feed element 0 to every MFMA.
  static __device__ __forceinline__ floatx4 mma_chunk(u32x4 a, u32x4 b, floatx4 c) {
    const floatx4 x = __builtin_bit_cast(floatx4, a), y = __builtin_bit_cast(floatx4, b);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(x[0], y[0], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(x[1], y[1], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(x[2], y[2], c, 0, 0, 0);
    c = __builtin_amdgcn_mfma_f32_16x16x4f32(x[3], y[3], c, 0, 0, 0);
    return c;
  }
  struct AFrag { float v[8]; };
  struct TFrag {
    float v[8];
    __device__ __forceinline__ void set(int i, float x) { v[i] = x; }
  };
  static __device__ __forceinline__ floatx4 mma_acc(const AFrag& a, const TFrag& b, floatx4 c) {
#pragma unroll
    for (int i = 0; i < 8; ++i) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a.v[i], b.v[i], c, 0, 0, 0);
    return c;
  }
  static __device__ __forceinline__ void store4(float* p, floatx4 x) { *(floatx4*)p = x; }
  static __device__ __forceinline__ floatx4 load4(const float* p) { return *(const floatx4*)p; }
  static __device__ __forceinline__ float dot_chunk(u32x4 a, u32x4 b) {
    const floatx4 x = __builtin_bit_cast(floatx4, a), y = __builtin_bit_cast(floatx4, b);
    return __builtin_fmaf(x[3], y[3], __builtin_fmaf(x[2], y[2], __builtin_fmaf(x[1], y[1], x[0] * y[0])));
  }
};

// ---------------------------------------------------------------------------
// LDS tile geometry.  A streamed tile is kBS rows x D elements, stored
// without padding; the 16-byte chunks of each row are permuted (slot =
// phys(r, c) for logical chunk c of row r) so that both LDS read patterns run
// without bank conflicts.  What gfx950 needs, as measured with the
// SQ_LDS_BANK_CONFLICT counter on probe patterns:
//   * ds_read_b128 (score A-operands; lane (g, j) reads row j, chunk 4kk+g):
//     within each group of 4 consecutive lanes the four 16-byte slots (mod
//     256 bytes) must form two aligned 32-byte pairs;
//   * ds_read_b64_tr_b16 (transposed accumulate operands; lane (g, j) reads 8
//     bytes of row 4g + j/4): the 32 lanes served together must hit 32
//     distinct 8-byte slots mod 256 bytes.
// A per-row XOR cannot satisfy both, so bf16 rows use the permutations below
// (row pairs share a 64-byte quad and differ in the low slot bit; successive
// row pairs rotate through the quads).  fp32 tiles are only read with
// ds_read_b128 and scalar loads and use slot = c ^ (r mod 16).
// ---------------------------------------------------------------------------
template <typename T, int D> struct Geo {
  static constexpr int kCPR = D * (int)sizeof(T) / 16;          // 16-byte chunks per row
  static constexpr int kChunks = D * (int)sizeof(T) / 64;       // score MFMA steps per row
  static constexpr int kEPC = 16 / (int)sizeof(T);              // elements per chunk
  static constexpr int kTileElems = kBS * D;                     // one streamed tile in LDS
  static constexpr int kNB = D / 16;                             // 16-dim output blocks
  static constexpr int kBlocks = kBS * kCPR / 64;                // 1 KB blocks per tile

  // physical slot of logical chunk c in row r (d = 64, 128; a d = 256 row
  // uses the d = 128 order in each of its 256-byte halves), and its inverse
  static __device__ __forceinline__ int phys(int r, int c) {
    if constexpr (sizeof(T) == 4) {
      return c ^ (r & (kCPR >= 16 ? 15 : kCPR - 1));
    } else if constexpr (D == 128) {
      return 4 * ((((r >> 1) & 3) + (c >> 1)) & 3) + 2 * (c & 1) + (((c >> 3) & 1) ^ (r & 1));
    } else if constexpr (D == 256) {
      return 16 * (c >> 4) +
             (4 * ((((r >> 1) & 3) + ((c & 15) >> 1)) & 3) + 2 * (c & 1) + (((c >> 3) & 1) ^ (r & 1)));
    } else {
      static_assert(D == 64, "head dim");
      return 4 * ((((r >> 2) & 1) + (c >> 1)) & 1) + 2 * (c & 1) + (((c >> 2) & 1) ^ ((r >> 1) & 1));
    }
  }
  static __device__ __forceinline__ int logical(int r, int p) {
    if constexpr (sizeof(T) == 4) {
      return p ^ (r & (kCPR >= 16 ? 15 : kCPR - 1));
    } else if constexpr (D == 128) {
      const int nb = (((p & 1) ^ (r & 1)) << 2) | (((p >> 2) - ((r >> 1) & 3)) & 3);
      return 2 * nb + ((p >> 1) & 1);
    } else if constexpr (D == 256) {
      const int q = p & 15;
      const int nb = (((q & 1) ^ (r & 1)) << 2) | (((q >> 2) - ((r >> 1) & 3)) & 3);
      return 16 * (p >> 4) + 2 * nb + ((q >> 1) & 1);
    } else {
      const int nb = (((p & 1) ^ ((r >> 1) & 1)) << 1) | ((p >> 2) ^ ((r >> 2) & 1));
      return 2 * nb + ((p >> 1) & 1);
    }
  }
  // d = 32 bf16 rows are only 64 bytes, so no permutation inside a row can
  // pair the slots of four consecutive rows: row pairs are interleaved at
  // 16-byte granularity instead (row 2i and 2i+1 share a 128-byte block,
  // chunk c of both side by side), and the chunk order rotates by two with
  // bit 2 of the row so the transposed reads stay on distinct slots.
  static constexpr bool kPairRows = sizeof(T) == 2 && D == 32;

  // element offset of logical chunk c of tile row r
  static __device__ __forceinline__ int chunk_off(int r, int c) {
    if constexpr (kPairRows)
      return kEPC * (8 * (r >> 1) + 2 * ((c + 2 * ((r >> 2) & 1)) & 3) + (r & 1));
    else
      return r * D + phys(r, c) * kEPC;
  }
  // inverse of chunk_off for the HBM -> LDS copy: the (row, chunk) whose 16
  // bytes belong at tile slot q
  static __device__ __forceinline__ void slot_source(int q, int& r, int& c) {
    if constexpr (kPairRows) {
      const int w = q & 7;
      r = 2 * (q >> 3) + (w & 1);
      c = ((w >> 1) - 2 * ((r >> 2) & 1)) & 3;
    } else {
      r = q / kCPR;
      c = logical(r, q % kCPR);
    }
  }

  // A-operand of the accumulate step: dims [dim0, dim0+16) x the 32 tile rows,
  // transposed; lane l gets rows {4g..4g+3, 16+4g..16+4g+3} (g = l >> 4) of
  // dim dim0 + (l & 15), matching the score tiles' row order.
  static __device__ __forceinline__ typename Elt<T>::AFrag load_afrag(const T FB_LDS* X, int dim0) {
    const int l = lane_id(), g = l >> 4, j = l & 15;
    typename Elt<T>::AFrag a;
    if constexpr (sizeof(T) == 2) {
      const int r = 4 * g + (j >> 2);
      const int c = (dim0 >> 3) + ((j & 3) >> 1);
      const int sub = 4 * (j & 1);
      shortx4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((shortx4 FB_LDS*)(X + chunk_off(r, c) + sub));
      shortx4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((shortx4 FB_LDS*)(X + chunk_off(r + 16, c) + sub));
      a.v = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
    } else {
      const int dim = dim0 + j;
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int r = 0; r < 4; ++r) a.v[4 * h + r] = X[chunk_off(16 * h + 4 * g + r, dim >> 2) + (dim & 3)];
    }
    return a;
  }
};

// Map a workgroup to (head, row block).  Workgroups are dispatched round-robin
// over the 8 XCDs; when the count allows it, consecutive logical blocks (which
// stream the same head's tensors) are kept on one XCD so they share its L2.
// With `reverse`, block indices run from the last block down (under a causal
// mask the last query blocks carry the most tiles, so they start first).
__device__ __forceinline__ void map_block(int nRB, int total, int& bh, int& rb, bool reverse = false) {
  int wg = blockIdx.x;
  int logical = ((total & 7) == 0) ? (wg & 7) * (total >> 3) + (wg >> 3) : wg;
  bh = logical / nRB;
  rb = logical - bh * nRB;
  if (reverse) rb = nRB - 1 - rb;
}

// How a streamed tile of kBS rows starting at s0 meets one wave's stationary
// rows [lo, hi] (N valid rows; causal mask: key <= query):
//   0 = no valid element (skip the tile's math), 1 = every element valid,
//   2 = mixed (mask per element).
// Row-major kernels: stationary = query rows, streamed = key rows.
__device__ __forceinline__ int tile_mode_rowmajor(int s0, int lo, int hi, int N, bool causal) {
  if (causal && s0 > hi) return 0;
  if (s0 + kBS <= N && (!causal || s0 + kBS - 1 <= lo)) return 1;
  return 2;
}
// Column-major kernels: stationary = key rows, streamed = query rows.
__device__ __forceinline__ int tile_mode_colmajor(int s0, int lo, int hi, int N, bool causal) {
  if (causal && s0 + kBS - 1 < lo) return 0;
  if (s0 + kBS <= N && (!causal || s0 >= hi)) return 1;
  return 2;
}


// Load the B-operand chunks of one stationary 16-row block: lane l holds row
// `row`, chunk kk = dims [kk*kKC + g*kKC/4, +kKC/4) with g = l >> 4.
// Rows >= N read 0.
template <typename T, int D, int NC>
__device__ __forceinline__ void load_stationary(u32x4 (&f)[NC], const T* head, int row, int N) {
  static_assert(NC == Geo<T, D>::kChunks, "chunk count");
  const int g = lane_id() >> 4;
#pragma unroll
  for (int kk = 0; kk < NC; ++kk) {
    if (row < N)
      f[kk] = *(const u32x4*)(head + (int64_t)row * D + kk * Elt<T>::kKC + g * (Elt<T>::kKC / 4));
    else
      f[kk] = u32x4{0u, 0u, 0u, 0u};
  }
}

// A streamed tile is copied HBM -> LDS in 1 KB blocks: each wave load
// instruction fills one contiguous block, lane i writing 16 bytes at offset
// 16*i, so the lane fetches the logical chunk that belongs at that (permuted)
// position (TileCopy below).  The copy is asynchronous: wait_vm<>() before
// the barrier that publishes it.
// Loads each wave issues per streamed tile: the NTENS x kBlocks 1 KB blocks
// of one tile stage are dealt out evenly over the NW waves.
template <typename T, int D, int NW, int NTENS>
constexpr int tile_loads() {
  static_assert((NTENS * Geo<T, D>::kBlocks) % NW == 0, "tile blocks per wave");
  return NTENS * Geo<T, D>::kBlocks / NW;
}

// The copy of NTENS streamed tiles by one of the NW waves that share it (w
// its index among them; TileCopy is built once, before the tile loop), with
// buffer_load ... lds.  Per tile and tensor the wave builds, in scalar
// registers, a buffer resource whose base is the tile's first row and whose
// size ends at row N; each lane's 32-bit byte offset into the tile (its
// chunk's row and column) is the same for every tile.  Issuing a tile
// therefore costs no vector address arithmetic, and rows at or past N read
// as zeros by the buffer's range check (finite data that every kernel masks
// out).
template <typename T, int D, int NW, int NTENS>
struct TileCopy {
  using G = Geo<T, D>;
  static constexpr int kBlockElems = 1024 / (int)sizeof(T);
  static constexpr bool kAllTensors = G::kBlocks % NW == 0;   // else kWPB waves share a block position
  static constexpr int kWPB = kAllTensors ? 1 : NW / G::kBlocks;
  static constexpr int kPos = kAllTensors ? G::kBlocks / NW : 1;   // block positions this wave copies
  static constexpr int kRowBytes = D * (int)sizeof(T);
  static_assert(kAllTensors || (NW % G::kBlocks == 0 && NTENS % kWPB == 0), "tile blocks per wave");
  int w;                       // wave-uniform
  uint32_t off[kPos];          // per-lane byte offset of the lane's chunk from the tile's first row

  __device__ __forceinline__ explicit TileCopy(int wave) {
    w = __builtin_amdgcn_readfirstlane(wave);
#pragma unroll
    for (int i = 0; i < kPos; ++i) {
      int r, c;
      G::slot_source(block(i) * 64 + lane_id(), r, c);
      off[i] = (uint32_t)(r * kRowBytes + c * 16);
    }
  }
  __device__ __forceinline__ int block(int i) const { return kAllTensors ? w + i * NW : w % G::kBlocks; }

  __device__ __forceinline__ void issue(const T* const (&src)[NTENS], T FB_LDS* dst, int s0, int N) const {
    // bytes from row s0 to the end of the tile or of the matrix (< 2^31)
    const int bytes = min(N - s0, kBS) * kRowBytes;
    auto one = [&](const T* base, int t, int i) {
#if defined(__HIP_DEVICE_COMPILE__)  // the buffer-resource type exists for the device target only
      const __amdgpu_buffer_rsrc_t rs =
          __builtin_amdgcn_make_buffer_rsrc((void*)(base + (int64_t)s0 * D), (short)0, bytes, 0x00020000);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          rs, (__attribute__((address_space(3))) void*)(dst + t * G::kTileElems + block(i) * kBlockElems), 16,
          off[i], 0, 0, 0);
#endif
    };
    if constexpr (kAllTensors) {
      // every wave takes the same block positions of every tensor
#pragma unroll
      for (int i = 0; i < kPos; ++i)
#pragma unroll
        for (int t = 0; t < NTENS; ++t) one(src[t], t, i);
    } else {
      // tensor index chosen by selects, not by indexing the pointer array
      // (which would go through scratch)
      const int t0 = w / G::kBlocks;
#pragma unroll
      for (int k = 0; k < NTENS / kWPB; ++k) {
        const int t = t0 + k * kWPB;
        const T* base = src[0];
#pragma unroll
        for (int u = 1; u < NTENS; ++u)
          if (t == u) base = src[u];
        one(base, t, 0);
      }
    }
  }
};

// Wait until at most N vector-memory loads of this wave are outstanding
// (loads complete in issue order for this count).
template <int N>
__device__ __forceinline__ void wait_vm() { asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory"); }


// Set the exponents of invalid (masked) tile entries to -inf, so exp2 gives
// P = 0 there.  x[sb][m][r] belongs to streamed row s0 + 16 sb + 4 (l >> 4) + r
// and stationary row t0 + 16 m, with t0 the lane's first stationary row.
// Row-major kernels (stationary = query t, streamed = key s): valid iff
// s < N and (no mask or s <= t).  Column-major kernels (stationary = key t,
// streamed = query s): valid iff s < N and (no mask or s >= t).
template <bool kRowMajor, int M>
__device__ __forceinline__ void mask_tile(floatx4 (&x)[2][M], int s0, int t0, int N, bool causal) {
  const int g = lane_id() >> 4;
#pragma unroll
  for (int sb = 0; sb < 2; ++sb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int sr = s0 + 16 * sb + 4 * g + r;
#pragma unroll
      for (int m = 0; m < M; ++m) {
        const int t = t0 + 16 * m;
        const bool ok = sr < N && (!causal || (kRowMajor ? sr <= t : sr >= t));
        x[sb][m][r] = ok ? x[sb][m][r] : -INFINITY;
      }
    }
}

// mask_tile for one stationary 16-row block: x[sb][r] belongs to streamed row
// s0 + 16 sb + 4 (l >> 4) + r and stationary row t.
template <bool kRowMajor>
__device__ __forceinline__ void mask_tile1(floatx4 (&x)[2], int s0, int t, int N, bool causal) {
  const int g = lane_id() >> 4;
#pragma unroll
  for (int sb = 0; sb < 2; ++sb)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int sr = s0 + 16 * sb + 4 * g + r;
      const bool ok = sr < N && (!causal || (kRowMajor ? sr <= t : sr >= t));
      x[sb][r] = ok ? x[sb][r] : -INFINITY;
    }
}

// The pipelined tile loop shared by every kernel: tiles it_begin .. it_end-1
// stream through an NSTAGE-deep LDS ring.  issue(tile, stage) starts the
// asynchronous copies of one tile (row scalars first, then the matrices, so
// that at most LT loads per wave are younger than the previous tile's);
// body(tile, stage) consumes a resident tile.  One barrier per tile.  The
// loop is unrolled by NSTAGE, so every ring-stage index the two callbacks
// see is a compile-time constant: LDS addresses become loop-invariant
// registers plus immediate offsets, and the copy's LDS destination a
// constant.
template <int NSTAGE, int LT, class Issue, class Body>
__device__ __forceinline__ void stream_loop(int it_begin, int it_end, Issue&& issue, Body&& body) {
  static_assert(NSTAGE == 2 || NSTAGE == 3, "pipeline depth");
  const int n = it_end - it_begin;
#pragma unroll
  for (int st = 0; st < NSTAGE - 1; ++st)
    if (st < n) issue(it_begin + st, st);
  wait_vm<0>();
  __syncthreads();
  // iteration k consumes stage k % NSTAGE and refills stage (k - 1) % NSTAGE
  auto step = [&](int k, auto cur) {
    constexpr int kCur = decltype(cur)::value;
    constexpr int kNext = kCur == 0 ? NSTAGE - 1 : kCur - 1;
    const int nx = k + NSTAGE - 1;  // tile fetched during this iteration
    if (nx < n) issue(it_begin + nx, kNext);
    body(it_begin + k, kCur);
    // the next tile must have landed; with three stages the one after it may
    // still be in flight
    if (NSTAGE == 3 && nx < n)
      wait_vm<LT>();
    else
      wait_vm<0>();
    __syncthreads();
  };
  for (int k = 0; k < n; k += NSTAGE) {
    step(k, std::integral_constant<int, 0>{});
    if (k + 1 < n) step(k + 1, std::integral_constant<int, 1>{});
    if constexpr (NSTAGE == 3)
      if (k + 2 < n) step(k + 2, std::integral_constant<int, 2>{});
  }
}
// stream_loop for a kernel that transforms the streamed row scalars once per
// tile before use.  One wave (`owner`) copies the scalars of tile t just
// before the matrices of tile t-1 (issue_s, LS loads), so they have landed
// by the time tile t-1 is consumed.  The body of tile t-1 calls prep_next()
// exactly once on every path (after its score MFMAs are issued, so that the
// owner's LDS round trip overlaps them): on the owner that runs prep(t), which
// reads the raw copy and writes the transformed values into the slot that
// tile t-2 used, and the barrier at the end of the iteration publishes them.
// issue_m(tile, matrix stage) issues LT loads per wave; issue_s(tile, scalar
// stage) and prep(tile, scalar stage, transformed slot) run on the owner only;
// body(tile, matrix stage, transformed slot, prep_next).  Two stages: the
// loop is unrolled by two, so every stage and slot index is a compile-time
// constant (as in stream_loop).
template <int NSTAGE, int LT, int LS, class IssueS, class IssueM, class Prep, class Body>
__device__ __forceinline__ void stream_loop_rs(int it_begin, int it_end, bool owner, IssueS&& issue_s,
                                               IssueM&& issue_m, Prep&& prep, Body&& body) {
  static_assert(NSTAGE == 2, "the column kernels run a two-stage ring");
  const int n = it_end - it_begin;
  if (owner && n > 0) issue_s(it_begin, 0);
  if (n > 0) {
    if (owner && 1 < n) issue_s(it_begin + 1, 1);
    issue_m(it_begin, 0);
  }
  wait_vm<0>();
  if (owner && n > 0) prep(it_begin, 0, 0);
  __syncthreads();
  // iteration k: matrices in stage k % 2 (the next tile's go to the other
  // stage), raw scalars of tile k + 2 into stage k % 2, transformed scalars of
  // tile k in slot k % 2
  auto step = [&](int k, auto cur) {
    constexpr int kCur = decltype(cur)::value, kOther = 1 - kCur;
    const int nx = k + 1;
    if (nx < n) {
      if (owner && nx + 1 < n) issue_s(it_begin + nx + 1, kCur);
      issue_m(it_begin + nx, kOther);
    }
    body(it_begin + k, kCur, kCur, [&]() {
      if (owner && k + 1 < n) prep(it_begin + k + 1, kOther, kOther);
    });
    // the next tile's matrices (and, on the owner, the scalars of the tile
    // after) must have landed
    wait_vm<0>();
    __syncthreads();
  };
  for (int k = 0; k < n; k += 2) {
    step(k, std::integral_constant<int, 0>{});
    if (k + 1 < n) step(k + 1, std::integral_constant<int, 1>{});
  }
}

// Iteration space of a column-major kernel's streaming loop.  The streamed
// side is the query tiles it_begin .. it_begin + nTh - 1 (under the causal
// mask the tiles before it_begin lie entirely above the column block's
// diagonal).  With kGQA it is those tiles of each of the grp query heads that
// share key/value head bh, one head after another: nIt = grp * nTh flattened
// iterations, flattened iteration i being tile it_begin + i % nTh of query
// head bh * grp + i / nTh.  With KS wave sets, set ks takes flattened
// iterations ks, ks + KS, ks + 2 KS, ...; every set runs the same number of
// loop iterations (the loop's barriers are workgroup-wide), and an iteration
// past the end (live() false) loads the last valid tile again and skips the
// math, so each wave's count of outstanding copies is the same as on a live
// iteration.  With kParts the column block is split over nparts workgroups
// (one wave set each): part p takes flattened iterations p, p + nparts, ...,
// and its loop simply runs that many iterations (none if p >= nIt).
template <bool kGQA, int KS, bool kParts = false>
struct StreamSplit {
  static_assert(!kParts || (KS == 1 && kGQA), "a split column block runs one wave set on the grouped loop");
  int it_begin, nTh, nIt, ks, bh, grp;
  int part = 0, nparts = 1;
  __device__ __forceinline__ int begin() const { return KS == 1 && !kGQA ? it_begin : 0; }
  __device__ __forceinline__ int end(int nT) const {
    if (kParts) return (nIt - part + nparts - 1) / nparts;
    return KS == 1 ? (kGQA ? nIt : nT) : (nIt + KS - 1) / KS;
  }
  __device__ __forceinline__ int flat(int it) const {
    if (kParts) return part + nparts * it;
    return KS == 1 ? it : min(ks + KS * it, nIt - 1);
  }
  __device__ __forceinline__ bool live(int it) const { return KS == 1 || ks + KS * it < nIt; }
  __device__ __forceinline__ int qhead(int it) const { return kGQA ? bh * grp + flat(it) / nTh : bh; }
  __device__ __forceinline__ int tile(int it) const {
    if (KS == 1 && !kGQA) return it;
    return it_begin + (kGQA ? flat(it) % nTh : flat(it));
  }
};

// Job numbering of a column kernel whose column blocks are split over
// nparts workgroups (grid = total * nparts, total = heads * nRB):
// job = (rb * heads + bh) * nparts + part.  Under the causal mask block rb
// holds work in proportion to the tiles at or below its diagonal, so jobs run
// heaviest first, and consecutive jobs (which the dispatcher sends to
// different XCDs) carry similar work.
__device__ __forceinline__ void map_column_job(int nRB, int total, int nparts, int& bh, int& rb, int& part) {
  const int heads = total / nRB, job = blockIdx.x;
  rb = job / (heads * nparts);
  const int rest = job - rb * heads * nparts;
  bh = rest / nparts;
  part = rest - bh * nparts;
}

// One part's fp32 sums of a split column kernel: x and y (the two key-side
// accumulators, [16-dim block][stationary sub-block]) of the lane's rows
// col0 + 16 m + (lane & 15) go to planes 2 part and 2 part + 1 of parts_out
// ([nparts][2][heads][N][D]), at head offset hoff.  Every part stores all
// of its rows, zeros included, so the reduction needs no cleared buffer.
template <int D, int NB, int MC>
__device__ __forceinline__ void store_column_part(float* parts_out, int64_t plane, int part, int64_t hoff,
                                                  int col0, int N, const floatx4 (&x)[NB][MC],
                                                  const floatx4 (&y)[NB][MC]) {
  const int l = lane_id(), g = l >> 4, j = l & 15;
  float* px = parts_out + 2 * (int64_t)part * plane;
  float* py = px + plane;
#pragma unroll
  for (int mc = 0; mc < MC; ++mc) {
    const int col = col0 + 16 * mc + j;
    if (col < N) {
#pragma unroll
      for (int nb = 0; nb < NB; ++nb) {
        const int64_t off = hoff + (int64_t)col * D + 16 * nb + 4 * g;
        *(floatx4*)(px + off) = x[nb][mc];
        *(floatx4*)(py + off) = y[nb][mc];
      }
    }
  }
}

// Two-level accumulation for the key-side sums of a column kernel (kOn).
// A column block's Kt/Vt (or dK/dV) sums run over every streamed query tile,
// G * N / 32 MFMA steps into one fp32 accumulator.  The MFMA's own fp32
// accumulation is not round-to-nearest: when the accumulator is far larger
// than one step's products it loses their low bits toward one side, and that
// one-signed error grows with the chain (measured: the zero column sums
// sum_j Kt_j = 0 drift from 3e-3 at N = 2^19 to 3e-2 at N = 2^21, and the
// residual falls in proportion to the chain when it is cut).  With kOn the
// MFMA chain runs `every` streamed tiles, is added into fp32 section sums
// by ordinary (round-to-nearest) VALU adds, and restarts from zero; finish()
// adds the last partial section.  x, y are [16-dim block][stationary block].
template <bool kOn, int A, int B>
struct SectionSums {
  floatx4 sx[kOn ? A : 1][kOn ? B : 1], sy[kOn ? A : 1][kOn ? B : 1];
  int n;
  __device__ __forceinline__ void init() {
    n = 0;
    if constexpr (kOn) {
#pragma unroll
      for (int a = 0; a < A; ++a)
#pragma unroll
        for (int b = 0; b < B; ++b) sx[a][b] = sy[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
  }
  // after the accumulate MFMAs of one streamed tile
  __device__ __forceinline__ void step(floatx4 (&x)[A][B], floatx4 (&y)[A][B], int every) {
    if constexpr (kOn) {
      if (++n == every) {
        n = 0;
#pragma unroll
        for (int a = 0; a < A; ++a)
#pragma unroll
          for (int b = 0; b < B; ++b) {
            sx[a][b] += x[a][b];
            sy[a][b] += y[a][b];
            x[a][b] = y[a][b] = floatx4{0.f, 0.f, 0.f, 0.f};
          }
      }
    }
  }
  __device__ __forceinline__ void finish(floatx4 (&x)[A][B], floatx4 (&y)[A][B]) {
    if constexpr (kOn) {
#pragma unroll
      for (int a = 0; a < A; ++a)
#pragma unroll
        for (int b = 0; b < B; ++b) {
          x[a][b] = sx[a][b] + x[a][b];
          y[a][b] = sy[a][b] + y[a][b];
        }
    }
  }
};

// Two wave sets of one workgroup that accumulated the same stationary rows
// over disjoint sets of streamed tiles: set 1 hands its fp32 accumulators x,
// then y, to set 0 through LDS (buf: every wave's A*B 1 KB blocks, placed by
// the wave's index wl within its set), and set 0 adds them, always in the
// order set 0 + set 1.  Every wave of the workgroup calls it (it holds
// barriers); buf may alias the tile ring once the streaming loop has ended
// (its last barrier follows the last read and the last copy).
template <int A, int B>
__device__ __forceinline__ void merge_wave_sets(floatx4 (&x)[A][B], floatx4 (&y)[A][B], int ks, int wl,
                                                floatx4 FB_LDS* buf) {
  floatx4 FB_LDS* p = buf + wl * (A * B * 64) + lane_id();
  auto one = [&](floatx4 (&acc)[A][B]) {
    if (ks == 1) {
#pragma unroll
      for (int a = 0; a < A; ++a)
#pragma unroll
        for (int b = 0; b < B; ++b) p[(a * B + b) * 64] = acc[a][b];
    }
    __syncthreads();
    if (ks == 0) {
#pragma unroll
      for (int a = 0; a < A; ++a)
#pragma unroll
        for (int b = 0; b < B; ++b) acc[a][b] += p[(a * B + b) * 64];
    }
  };
  one(x);
  __syncthreads();  // set 0 has read x before set 1 overwrites it with y
  one(y);
}

// Streamed per-row fp32 scalars (L, D, alpha, E) for one tile, copied HBM ->
// LDS with global_load_lds_dword: one wave instruction moves two kBS-float
// vectors (lanes 0..31 read `a`, lanes 32..63 read `b`) to dst[0 .. 63].
// Indices >= N are clamped to N-1; the kernels mask those rows.  The two base
// pointers are passed by value so that the per-lane choice is a register
// select (an indexed pointer array would go through scratch memory and force
// a full vmcnt wait).  Asynchronous like the tile copy.
__device__ __forceinline__ void issue_scalar_pair(float FB_LDS* dst, const float* a, const float* b, int s0, int N) {
  static_assert(kBS == 32, "two 32-float vectors per wave instruction");
  const int l = lane_id();
  const int idx = min(s0 + (l & 31), N - 1);
  const float* p = (l < 32 ? a : b) + idx;
  __builtin_amdgcn_global_load_lds((const __attribute__((address_space(1))) void*)p,
                                   (__attribute__((address_space(3))) void*)dst, 4, 0, 0);
}

}  // namespace fb
