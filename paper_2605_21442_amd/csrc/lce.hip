// liblce: linear-cross-entropy (LCE) forward and backward for MI355X (gfx950).
//
// The objective is the paper's Linear Cross-Entropy loss (Sec. 4.2): the final
// output projection H W^T is fused with the cross-entropy over the whole
// vocabulary, ignored targets are dropped before the projection, and the dense
// [tokens, vocab] logits never exist. The result equals the standard
// cross-entropy (Sec. 3.3). The ABI, its conventions and its error codes are
// documented in include/lce.h.
//
// Path (all kernels enqueue on the caller's stream, no host synchronisation):
//   forward : compact -> gather the valid rows Hv -> fwd_tile (bf16 MFMA tiles of
//             S^T = W Hv^T, each reduced to a (max, sum-exp) partial per token) ->
//             combine (merge partials, target logit, per-row loss) -> loss (fixed-order
//             reduction)
//   backward: compact -> gather Hv (both skipped when the forward's are reused) -> per
//             vocabulary slab: G tile (recompute S^T, G = c (softmax - onehot)),
//             dH32 (+)= G W_slab (K split into parts where a launch would leave CUs idle),
//             dW slab = G^T Hv -> finalise dH (parts added in order)
// Built on the same kernels: the backward with an AdamW step on each finished dW block
// (paper Sec. 4.1), a vocabulary-shard (loss-parallel) forward / combine / backward, and a
// fused linear knowledge-distillation loss whose G kernel takes the teacher's probabilities
// as soft targets.
//
// Every contraction C = A B^T (C [M, N], sum over K) runs one MFMA main loop: bf16
// v_mfma_f32_32x32x16 with fp32 accumulation, waves of 128x64 outputs, K streamed through
// two 64-wide LDS slices filled by direct-to-LDS buffer loads (XOR-swizzled 16-byte
// chunks). Tiles are 384x256 with 12 waves (three per SIMD) for the LCE contractions when
// D % 64 == 0, else 256x256 with 8 waves. Each operand is either K-contiguous (W and Hv in
// the forward and G kernels; G in dH) or K-major (G and Hv in dW, the W slab in dH: the
// MFMA fragments then come from transposing LDS reads), so G is written once, token-major,
// and W is never copied.
//
// Launch shapes follow the 8 XCDs, each with its own L2 (workgroups are dealt to them round-
// robin): the forward and G tiles go in vocabulary groups a multiple of 8 tiles wide, so that each
// XCD keeps its own W tiles while the token tiles pass (xcd_tile); the dH and dW tiles are cut into
// balanced per-XCD shares walked in bands of 4 row tiles; and the backward slab width is chosen so
// that the dW launches fill whole rounds of the 256 CUs (whole_round_slab).

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <type_traits>
#include <utility>
#include <vector>

#include "lce.h"

// Workspace of lce_forward_noalloc: device memory of the code object itself, one copy per GPU,
// held until the process ends. In host code `scratch` is only a stand-in for the symbol; its
// device address comes from hipGetSymbolAddress (see noalloc_scratch).
static __device__ __align__(256) char scratch[LCE_NOALLOC_SCRATCH_BYTES];

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef int i32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
typedef short s16x4_t __attribute__((ext_vector_type(4)));
typedef short s16x8_t __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) s16x4_t lds_s16x4_t;

constexpr int TILE = 256;         // output tile edge (rows of A and of B per workgroup)
constexpr int KPAD = 64;          // K padding granularity of the backward's staged operands
constexpr int NTHREADS = 512;     // 8 waves, two per SIMD
constexpr int MAX_PARTS = 32;     // vocabulary partitions of the forward (x2 wave rows <= 64 lanes)
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr uint32_t kRsrcWord3 = 0x00020000u;  // gfx9 raw buffer: 32-bit data format

// Raw buffer descriptor: base address, stride 0, num_records = bytes. num_records is capped below
// 2^31 so that offset 2^31 is always out of range (the zero-fill trick for ragged K slices); every
// access of a tile lies within its first 2^31 bytes (checked on the host, or the descriptor is
// rebuilt per slice). Two forms: the compiler's buffer-resource type for the load builtin, and the
// 4 descriptor words (in SGPRs) for the inline-asm load.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint64_t bytes) {
  const uint32_t n = bytes > 0x7FFFFFFFull ? 0x7FFFFFFFu : (uint32_t)bytes;
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)n, (int)kRsrcWord3);
}

__device__ __forceinline__ i32x4_t make_rsrc_words(const void* base, uint64_t bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  const uint32_t n = bytes > 0x7FFFFFFFull ? 0x7FFFFFFFu : (uint32_t)bytes;
  i32x4_t w;
  w.x = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
  w.y = __builtin_amdgcn_readfirstlane((int)((a >> 32) & 0xFFFFu));
  w.z = __builtin_amdgcn_readfirstlane((int)n);
  w.w = (int)kRsrcWord3;
  return w;
}

typedef __attribute__((address_space(3))) void lds_void_t;

// One direct-to-LDS load: 16 bytes per lane from the buffer at voffset + soffset into LDS at lds
// + 16 * lane (lds wave-uniform; m0 is its LDS byte address).
//  kAsm = false: the compiler builtin. The compiler tracks it as an LDS write and, before any LDS
//    read it cannot prove disjoint, waits for every such load in flight; it proves this for the
//    128-bit fragment reads but not for the transposing reads.
//  kAsm = true: inline asm, which the compiler does not track, for the main loops that use
//    transposing reads (a compiler wait there would stall each substep on the next slice's
//    loads). The main loop orders the loads against the reads itself: a vmcnt wait and a barrier
//    before a buffer is read, and a buffer is refilled only after the barrier that follows its
//    last read. The s_nop is the wait state an M0 write needs before a load that writes LDS.
template <bool kAsm>
__device__ __forceinline__ void dma16(const __amdgpu_buffer_rsrc_t& rs, const i32x4_t& rw, const char* lds, int m0,
                                      uint32_t voffset, uint32_t soffset) {
  if constexpr (!kAsm) {
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)lds, 16, (int)voffset, (int)soffset, 0, 0);
  } else {
    // m0 is an input operand: the compiler sets it (and knows the value it holds afterwards)
    asm volatile("s_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
                 :
                 : "v"(voffset), "s"(rw), "s"(soffset), "{m0}"(m0)
                 : "memory");
  }
}

// A 16-byte global store followed by 8 wait states, in one statement. On this part a store wider
// than 8 bytes reads its data registers after it issues, and rewriting them within a few
// instructions corrupts the stored data, while the compiler keeps only one wait state there; the
// padding keeps the next instructions of the wave away from the data registers.
__device__ __forceinline__ void store16_padded(void* p, i32x4_t v) {
  asm volatile("global_store_dwordx4 %0, %1, off\n\ts_nop 7" : : "v"(p), "v"(v) : "memory");
}

// The same for a 16-byte store through a buffer resource (descriptor words rw, per-lane voffset,
// uniform soffset).
__device__ __forceinline__ void buffer_store16_padded(i32x4_t v, const i32x4_t& rw, uint32_t voffset,
                                                      uint32_t soffset) {
  asm volatile("buffer_store_dwordx4 %0, %1, %2, %3 offen\n\ts_nop 7"
               :
               : "v"(v), "v"(voffset), "s"(rw), "s"(soffset)
               : "memory");
}

__device__ __forceinline__ float bf16_to_f32(uint32_t bits16) { return __uint_as_float(bits16 << 16); }

// two floats rounded to nearest-even bf16 in one packed conversion (lo in the low half)
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

__device__ __forceinline__ uint16_t to_bf16(float x) { return __builtin_bit_cast(uint16_t, (__bf16)x); }

// ---------------------------------------------------------------------------------------------
// AdamW (decoupled weight decay, bias-corrected moments): the optimizer that paper Sec. 4.1
// runs inside the backward pass. The per-call constants are formed once on the host; the
// element update is one function shared by the fused dW epilogue and the standalone step, with
// floating-point contraction off so both give the same bits.
// ---------------------------------------------------------------------------------------------
struct AdamWConst {
  float keep;           // 1 - lr * weight_decay
  float beta1, omb1;    // beta1, 1 - beta1
  float beta2, omb2;    // beta2, 1 - beta2
  float step_size;      // lr / (1 - beta1^t)
  float inv_sqrt_bc2;   // 1 / sqrt(1 - beta2^t)
  float eps;
};

// Parameter and moments of W [V, D]: W bf16 with row stride ldw; m, v (and master, if not null)
// fp32 dense with row stride d.
struct AdamWState {
  uint16_t* W;
  int64_t ldw;
  float* m;
  float* v;
  float* master;
};

__device__ __forceinline__ void adamw_update(float& p, float& m, float& v, float g, const AdamWConst& c) {
#pragma clang fp contract(off)
  p = p * c.keep;
  m = c.beta1 * m + c.omb1 * g;
  v = c.beta2 * v + c.omb2 * (g * g);
  const float denom = sqrtf(v) * c.inv_sqrt_bc2 + c.eps;
  p = p - c.step_size * (m / denom);
}

__device__ __forceinline__ int64_t load_target(const void* t, int tbytes, int64_t i) {
  return tbytes == 8 ? ((const int64_t*)t)[i] : (int64_t)((const int32_t*)t)[i];
}

__device__ __forceinline__ float wave_sum(float x) {
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m);
  return x;
}
// ---------------------------------------------------------------------------------------------
// MFMA main loop: acc[bi][bj] = A[128 WM x K] * B[256 x K]^T for this workgroup's (128 WM) x 256
// tile, WM = 2 (256 x 256, 8 waves, two per SIMD) or WM = 3 (384 x 256, 12 waves, three per SIMD;
// the waves of a SIMD cover each other's memory stalls with their MFMAs).
//
// The waves form a WM x 4 grid; wave w = 4 wr + wc owns output rows wr*128.. (A rows) and
// columns wc*64.. (B rows). acc[bi][bj] (bi < 4, bj < 2) is the 32x32 block (bi, bj) of that
// 128x64 wave tile; lane l, register r of a block holds row 8 (r / 4) + 4 (l / 32) + r % 4,
// column l % 32. A fragment for v_mfma_f32_32x32x16_bf16 is 8 consecutive K values of one row
// (lane l: row l % 32, K chunk l / 32 of the 16-wide substep).
//
// K streams through two LDS buffers of 64-wide slices (A 32 or 48 KB and B 32 KB per buffer),
// copied global -> LDS by buffer loads that write LDS directly, one 16-byte chunk per lane and
// 1 KB per instruction. An operand is stored in one of two ways:
//
//  * row-major (K contiguous, e.g. H [N, D], W [V, D]): a slice is 256 or 384 rows x 128 bytes; each
//    load instruction moves 8 rows (one full cache line per row, which the memory pipeline turns
//    into whole-line requests). Chunk c of row r sits at position c ^ swz(r), swz(r) = (r & 7) ^
//    ((r >> 3) & 1), so that the 128-bit fragment reads of any 8 or 16 consecutive rows hit
//    distinct banks;
//  * K-major (the tile's 256 or 384 elements contiguous, e.g. G [Nv, Vc] as the A operand of
//    G^T H, or W [V, D] as the B operand of G W): a slice is 64 K-rows x 512 or 768 bytes; each
//    load instruction moves whole lines of consecutive K-rows. For a 256-wide operand chunk c of
//    K-row k sits at position c ^ kswz(k), kswz(k) = 4 (k & 3) + 16 ((k >> 3) & 1) (the 384-wide
//    swizzle is kpos below). Fragments come from pairs of transposing reads
//    (ds_read_b64_tr_b16): in a 16-lane group, lane i reads 4 consecutive elements (8 bytes) of
//    K-row i / 4 and lane j receives element j of the group's 16 columns from K-rows 0..3; the
//    second read covers K-rows 4..7. The swizzle spreads the 4 K-rows x 64 bytes that a half-wave
//    reads over all banks.
//
// Each load picks its source chunk so that it lands in the swizzled position.
//
// Schedule of slice j (four 16-wide substeps; WM = 2 reads fragments one substep ahead, WM = 3
// just before use): after the third substep's MFMAs are issued, one barrier both publishes slice
// j+1 (its loads were issued about a slice earlier) and frees slice j's buffer, into which slice
// j+2 is then loaded while the fourth substep runs. Waves 0..3 issue their loads at the barrier,
// the others one or two substeps later (kLateGroups): on this part a whole workgroup's load
// instructions at once fill the texture-address queues and stall the issuing waves (measured:
// 3-9 % per kernel; the better delay depends on the operand stream).
//
// K must be a multiple of 8; a ragged last slice is zero-filled by pointing the lanes past K
// outside the buffer resource (buffer loads return 0 there).
// ---------------------------------------------------------------------------------------------
constexpr int KSLICE = 64;
constexpr uint32_t kOobOffset = 0x80000000u;

// Tile geometry of the main loop with WM wave rows: the A tile has 128 WM rows (256 or 384), the
// B tile 256; 4 WM waves (2 or 3 per SIMD). A slice buffer holds the A region (128 WM rows x 128
// bytes) followed by the B region (32 KB); two buffers.
template <int WM>
struct Geo {
  static constexpr int TM = 128 * WM;
  static constexpr int NT = 256 * WM;
  static constexpr int AREG = TM * 128;
  static constexpr int SLICE = AREG + 32768;
  static constexpr int LDS = 2 * SLICE;
};
constexpr int LDS_BYTES = Geo<2>::LDS;
constexpr int kDhWM = 3;   // wave rows of the dH contraction
constexpr int kDwWM = 3;   // wave rows of the dW contraction
constexpr int kGWM = 3;    // wave rows of the (one-hot) G kernel

// One operand of the main loop, kW (256 or 384) tile rows (row-major) or tile columns (K-major)
// wide. Waves w < kW / 32 load it, 4 KB of the operand's region per wave and slice; the load of
// the q-th kilobyte reads at voffset off[.] + soffset.
//  OP_DENSE:  rsrc covers the tile's rows (rows past the tile's end read as zeros); off[0] is
//             the byte offset of row w*32 + lane/8 plus this lane's even-q chunk (odd q: the
//             neighbouring lane's); row 8q adds q * qstride (scalar) and the slice's K offset
//             2 k0 (scalar).
//  OP_GATHER: rsrc covers the source buffer; off[q] is the byte offset of the gathered row plus
//             the chunk; the K offset is added as a scalar.
//  OP_KMAJOR: base points at K-row 0, first column of the tile; rows are ld elements apart and
//             the buffer holds `bytes` bytes from base on; the buffer resource is rebuilt per slice
//             at base + k0 * ld, so offsets stay small for any buffer size. kW = 256: off[0] /
//             off[1] are the offsets for q = 0 / 1, and q = 2 / 3 read 2 qstride (four K-rows)
//             further; kW = 384: off[q] per q.
struct Operand {
  __amdgpu_buffer_rsrc_t rsrc;
  i32x4_t rwords;
  const uint16_t* base;
  int64_t ld;
  uint64_t bytes;
  uint32_t off[4];
  uint32_t qstride;
};

// How an operand is stored: row-major rows of a dense buffer, row-major rows gathered through a
// row list, or K-major.
enum OpKind { OP_DENSE = 0, OP_GATHER = 1, OP_KMAJOR = 2 };

struct FragSet {
  bf16x8_t a[4], b[2];
};

// chunk this lane loads for its even-numbered rows (odd rows: ^ 1), row-major operands
__device__ __forceinline__ int lane_chunk_even() {
  const int j = threadIdx.x & 63;
  return (j & 7) ^ ((j >> 3) & 7);
}

// K-major swizzle: position in LDS of 16-byte chunk c (of kW / 8) of K-row k, and its inverse.
//  kW = 256: c ^ (4 (k & 3) + 16 ((k >> 3) & 1));
//  kW = 384: within each group of 16 chunks c ^ 4 (k & 3), and the three groups rotated by one
//            for K-rows with bit 3 set.
// Either way the 4 K-rows x 64 bytes a half-wave reads in one transposing read land on all banks.
__device__ __forceinline__ int kswz(int k) { return ((k & 3) << 2) | (((k >> 3) & 1) << 4); }

template <int kW>
__device__ __forceinline__ int kpos(int k, int c) {
  if constexpr (kW == 256) {
    return c ^ kswz(k);
  } else {
    const int g = (c >> 4) + ((k >> 3) & 1);
    return 16 * (g >= 3 ? g - 3 : g) + ((c & 15) ^ ((k & 3) << 2));
  }
}

template <int kW>
__device__ __forceinline__ int kchunk(int k, int pos) {
  if constexpr (kW == 256) {
    return pos ^ kswz(k);
  } else {
    const int g = (pos >> 4) - ((k >> 3) & 1);
    return 16 * (g < 0 ? g + 3 : g) + ((pos & 15) ^ ((k & 3) << 2));
  }
}

// LDS byte offset, within a kW-wide K-major operand region, of this lane's first transposing read
// for the 32-column block starting at column c0 of substep 0 (the second read is 8 kW bytes
// further: 4 K-rows; substep ks adds 32 kW ks: 16 K-rows).
template <int kW>
__device__ __forceinline__ uint32_t kmajor_frag_addr(int c0) {
  const int lane = threadIdx.x & 63, g = lane >> 4, i = lane & 15;
  const int k = 8 * (g >> 1) + (i >> 2);
  const int col = c0 + 16 * (g & 1) + 4 * (i & 3);
  return (uint32_t)(k * kW * 2 + (kpos<kW>(k, col >> 3) << 4) + (col & 7) * 2);
}

template <int kW>
__device__ __forceinline__ bf16x8_t read_tr_pair(const char* p) {
  s16x8_t t;
  t.lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)p);
  t.hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_t*)(p + 8 * kW));
  return __builtin_bit_cast(bf16x8_t, t);
}

// Per-lane LDS read addresses of one operand.
//  row-major: rk = row base | chunk of substep 0; substep ks reads at rk ^ 32 ks (the chunk index
//             (2 ks + lane / 32) ^ swz is the substep-0 chunk ^ 2 ks), block b 4096 b further.
//  K-major:   tr for block 0 (+ 32 kW ks per substep); block b (32 columns further) reads at
//             tr ^ (b << 6): within a wave's 128 or 64 columns the block index only changes bits
//             2-3 of the chunk index, which both swizzles keep as an XOR.
template <int kBlocks>
struct FragAddr {
  uint32_t rk;
  uint32_t tr;
};

template <bool kKM, int kW, int kBlocks>
__device__ __forceinline__ void frag_addr(FragAddr<kBlocks>& fa, int row0) {
  const int lane = threadIdx.x & 63;
  if constexpr (!kKM) {
    const int swz = (lane & 7) ^ ((lane >> 3) & 1);
    fa.rk = (uint32_t)((row0 + (lane & 31)) * 128) | (uint32_t)(((lane >> 5) ^ swz) * 16);
  } else {
    fa.tr = kmajor_frag_addr<kW>(row0);
  }
}

template <bool kKM, int kW, int kBlocks>
__device__ __forceinline__ void read_operand(bf16x8_t (&f)[kBlocks], const char* reg, const FragAddr<kBlocks>& fa,
                                             int ks) {
  if constexpr (!kKM) {
    // the base address is made opaque at each read, so that its per-substep variants are formed
    // next to the reads (one VALU op each) instead of being held in registers through the loop
    uint32_t rk = fa.rk;
    asm volatile("" : "+v"(rk));
    const char* p = reg + (rk ^ (uint32_t)(32 * ks));
#pragma unroll
    for (int b = 0; b < kBlocks; ++b) f[b] = *reinterpret_cast<const bf16x8_t*>(p + b * 4096);
  } else {
#pragma unroll
    for (int b = 0; b < kBlocks; ++b) f[b] = read_tr_pair<kW>(reg + (fa.tr ^ (uint32_t)(b << 6)) + ks * 32 * kW);
  }
}

__device__ __forceinline__ void mma_substep(f32x16_t (&acc)[4][2], const FragSet& f) {
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f.a[i], f.b[j], acc[i][j], 0, 0, 0);
}

// This wave's 4 load instructions of one kW-wide operand's slice k0 (dstp = the operand's region
// + 4 KB per wave, dst its LDS byte address). Lanes that must read zeros (past K on a ragged last
// slice) point outside the buffer resource.
template <bool kAsm, int kKind, int kW, bool kMasked>
__device__ __forceinline__ void load_operand(const Operand& op, const char* dstp, int dst, int k0, int K) {
  if constexpr (kKind != OP_KMAJOR) {
    const int ce = lane_chunk_even();
    // dense: the odd-q offset of lane L is the even-q offset of lane L ^ 1 (same row, the chunk
    // with the other parity), fetched by a quad swap instead of held in a register
    const uint32_t odd = kKind == OP_DENSE ? (uint32_t)__builtin_amdgcn_mov_dpp((int)op.off[0], 0xB1, 0xF, 0xF, false) : 0u;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const bool ok = !kMasked || k0 + (ce ^ (q & 1)) * 8 < K;
      const uint32_t v = kKind == OP_DENSE ? ((q & 1) ? odd : op.off[0]) : op.off[q];
      const uint32_t so = (uint32_t)k0 * 2 + (kKind == OP_DENSE ? (uint32_t)q * op.qstride : 0u);
      dma16<kAsm>(op.rsrc, op.rwords, dstp + q * 1024, dst + q * 1024, ok ? v : kOobOffset, so);
    }
  } else {
    const uint16_t* base = op.base + (int64_t)k0 * op.ld;
    const uint64_t bytes = op.bytes - (uint64_t)k0 * op.ld * 2;
    const __amdgpu_buffer_rsrc_t rs = make_rsrc(base, bytes);
    const i32x4_t rw = make_rsrc_words(base, bytes);
    const int p0 = (threadIdx.x >> 6) * 256 + (threadIdx.x & 63);   // 16-byte unit of q = 0
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const bool ok = !kMasked || k0 + (p0 + 64 * q) / (kW / 8) < K;
      const uint32_t v = kW == 256 ? op.off[q & 1] : op.off[q];
      const uint32_t so = kW == 256 ? (uint32_t)(q & 2) * op.qstride : 0u;   // off[1] holds q = 1's rows
      dma16<kAsm>(rs, rw, dstp + q * 1024, dst + q * 1024, ok ? v : kOobOffset, so);
    }
  }
}

// w: this wave's index in the workgroup, a wave-uniform (scalar) value
template <bool kAsm, int kAKind, int kBKind, int WM, bool kMasked>
__device__ __forceinline__ void load_slice(const Operand& A, const Operand& B, const char* buf, int bufoff, int k0,
                                           int K, int w) {
  const char* dstp = buf + w * 4096;
  const int dst = bufoff + w * 4096;   // LDS byte address (asm loads)
  load_operand<kAsm, kAKind, Geo<WM>::TM, kMasked>(A, dstp, dst, k0, K);
  if (WM == 2 || w < 8) load_operand<kAsm, kBKind, 256, kMasked>(B, dstp + Geo<WM>::AREG, dst + Geo<WM>::AREG, k0, K);
}

// s_waitcnt with only the vector-memory counter constrained (expcnt / lgkmcnt left at max)
#define LCE_WAIT_VM(n) __builtin_amdgcn_s_waitcnt((((n) & 15) | (7 << 4) | (15 << 8) | (((n) >> 4) << 14)))

// acc = A B^T for this workgroup's (128 WM) x 256 tile. WM = 2: 8 waves, fragments double-
// buffered (read one substep ahead). WM = 3: 12 waves (three per SIMD), 384 A rows, fragments
// single-buffered (the 168 registers a wave may hold at three waves per SIMD leave no room for a
// second set; the other two waves of the SIMD cover the read latency).
template <int kLateGroups, int kAKind = OP_DENSE, int kBKind = OP_GATHER, int WM = 2, bool kRagged = true>
__device__ __forceinline__ void mma_mainloop(f32x16_t (&acc)[4][2], const Operand& A, const Operand& B, int K,
                                             char* smem) {
  using G = Geo<WM>;
  constexpr bool kAKM = kAKind == OP_KMAJOR, kBKM = kBKind == OP_KMAJOR;
  const int wave = threadIdx.x >> 6;
  const int wr = wave >> 2, wc = wave & 3;
  FragAddr<4> fa;
  FragAddr<2> fb;
  frag_addr<kAKM, G::TM>(fa, wr * 128);
  frag_addr<kBKM, 256>(fb, wc * 64);
  auto read_frags = [&](FragSet& f, const char* buf, int ks) {
    read_operand<kAKM, G::TM>(f.a, buf, fa, ks);
    read_operand<kBKM, 256>(f.b, buf + G::AREG, fb, ks);
  };

#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = (f32x16_t){};

  const int S = (K + KSLICE - 1) / KSLICE;
  if (S <= 0) return;
  // kRagged = false: the caller guarantees K % 64 == 0
  const bool ragged = kRagged && (K % KSLICE) != 0;
  // loads as inline asm where transposing reads are used (see dma16)
  constexpr bool kAsm = kAKM || kBKM;
  const int lds0 = kAsm ? __builtin_amdgcn_readfirstlane((int)(uint32_t)(uintptr_t)smem) : 0;
  // One scalar copy of the wave index for the whole loop. Opaque to the compiler, so that it is
  // not recomputed from the work-item id register inside the loop: under register pressure that
  // register is spilled, and its reload would wait for every load in flight.
  int wsc = __builtin_amdgcn_readfirstlane(wave);
  asm volatile("" : "+s"(wsc));
  auto load = [&](int s) {
    char* buf = smem + (s & 1) * G::SLICE;
    const int bufoff = lds0 + (s & 1) * G::SLICE;
    if (ragged && s == S - 1) load_slice<kAsm, kAKind, kBKind, WM, true>(A, B, buf, bufoff, s * KSLICE, K, wsc);
    else load_slice<kAsm, kAKind, kBKind, WM, false>(A, B, buf, bufoff, s * KSLICE, K, wsc);
  };

  // waves of a 12-wave workgroup past the eighth load only A: 4 loads per slice instead of 8
  const bool a_only = WM == 3 && wsc >= 8;
  load(0);
  if (S > 1) {
    load(1);
    if (a_only) LCE_WAIT_VM(4);
    else LCE_WAIT_VM(8);
  } else {
    LCE_WAIT_VM(0);
  }
  __builtin_amdgcn_s_barrier();

  // Waves 0..3 (the first wave of each SIMD) issue their share of a slice's loads at the barrier;
  // the others kLateGroups MFMA substeps later: a smaller load burst, and the other waves of each
  // SIMD go straight back to MFMA work.
  // slot of this wave's loads: 0 at the barrier, 1 after the slice's last substep, 2 after the
  // next slice's first substep. kLateGroups = 1 or 2: waves 4.. use that slot; 1xy (WM = 3):
  // waves 4..7 use slot x, waves 8..11 slot y.
  constexpr int kMid = kLateGroups >= 100 ? (kLateGroups / 10) % 10 : kLateGroups;
  constexpr int kLast = kLateGroups >= 100 ? kLateGroups % 10 : kLateGroups;
  const int slot = wsc < 4 ? 0 : (WM == 3 && wsc >= 8 ? kLast : kMid);
  const bool late = slot != 0;
  int pend = -1;
  if constexpr (WM == 2) {
    FragSet f0, f1;
    read_frags(f0, smem, 0);
    for (int j = 0; j < S; ++j) {
      const char* cur = smem + (j & 1) * G::SLICE;
      const char* nxt = smem + ((j + 1) & 1) * G::SLICE;
      read_frags(f1, cur, 1);
      mma_substep(acc, f0);
      if (slot == 2 && pend >= 0) {
        load(pend);
        pend = -1;
      }
      read_frags(f0, cur, 2);
      mma_substep(acc, f1);
      read_frags(f1, cur, 3);
      mma_substep(acc, f0);
      if (j + 1 < S) {
        // slice j+1 landed (own loads) and every wave is done with slice j's buffer
        __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_s_barrier();
        if (j + 2 < S) {
          if (!late) load(j + 2);
          else pend = j + 2;
        }
        read_frags(f0, nxt, 0);
      }
      mma_substep(acc, f1);
      if (slot == 1 && pend >= 0) {
        load(pend);
        pend = -1;
      }
    }
  } else {
    FragSet f;
    for (int j = 0; j < S; ++j) {
      const char* cur = smem + (j & 1) * G::SLICE;
      read_frags(f, cur, 0);
      mma_substep(acc, f);
      if (slot == 2 && pend >= 0) {
        load(pend);
        pend = -1;
      }
      read_frags(f, cur, 1);
      mma_substep(acc, f);
      read_frags(f, cur, 2);
      mma_substep(acc, f);
      read_frags(f, cur, 3);
      if (j + 1 < S) {
        // slice j+1 landed (own loads) and every wave is done with slice j's buffer
        __builtin_amdgcn_s_waitcnt(0);
        __builtin_amdgcn_s_barrier();
        if (j + 2 < S) {
          if (!late) load(j + 2);
          else pend = j + 2;
        }
      }
      mma_substep(acc, f);
      if (slot == 1 && pend >= 0) {
        load(pend);
        pend = -1;
      }
    }
  }
  // every wave is done reading LDS before the caller reuses it
  __syncthreads();
}

// A row-major operand of rows [row0, row0 + kW) (tile = row0's start) of a dense buffer with
// rows_left rows from row0 on.
__device__ __forceinline__ Operand dense_operand(const uint16_t* tile, int rows_left, int64_t ld) {
  Operand op;
  op.rsrc = make_rsrc(tile, (uint64_t)rows_left * ld * 2);
  op.rwords = make_rsrc_words(tile, (uint64_t)rows_left * ld * 2);
  const int j = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int ce = lane_chunk_even();
  const uint32_t row = (uint32_t)((int64_t)(w * 32 + (j >> 3)) * ld * 2);
  op.off[0] = row + ce * 16;
  op.qstride = (uint32_t)(16 * ld);   // 8 rows
  return op;
}

// kW rows n0.. of the compacted valid-row list idx[0..nv) of a buffer of n rows (rows past nv
// repeat the last valid one).
template <int kW = 256>
__device__ __forceinline__ Operand gather_operand(const uint16_t* src, int64_t n, int64_t ld, const int* idx, int n0,
                                                  int nv) {
  Operand op;
  op.rsrc = make_rsrc(src, (uint64_t)n * ld * 2);
  op.rwords = make_rsrc_words(src, (uint64_t)n * ld * 2);
  const int j = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int ce = lane_chunk_even();
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    int r = w * 32 + q * 8 + (j >> 3);
    r = n0 + (r < kW ? r : kW - 1);
    r = r < nv ? r : nv - 1;
    op.off[q] = (uint32_t)((int64_t)idx[r] * ld * 2 + (ce ^ (q & 1)) * 16);
  }
  return op;
}

// The kW rows of a row-major tile (tile = its first row) of which only the first rows_left exist,
// e.g. the last vocabulary tile of W: per-row offsets as for a gathered operand (kind OP_GATHER),
// with the rows at or past rows_left pointed at kOobOffset. No address past the existing rows is
// formed, and the loads of the missing rows return zeros.
template <int kW>
__device__ __forceinline__ Operand masked_dense_operand(const uint16_t* tile, int rows_left, int64_t ld) {
  Operand op;
  op.rsrc = make_rsrc(tile, (uint64_t)rows_left * ld * 2);
  op.rwords = make_rsrc_words(tile, (uint64_t)rows_left * ld * 2);
  const int j = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int ce = lane_chunk_even();
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    int r = w * 32 + q * 8 + (j >> 3);
    r = r < kW ? r : kW - 1;   // (waves that do not load this operand)
    op.off[q] = r < rows_left ? (uint32_t)((int64_t)r * ld * 2 + (ce ^ (q & 1)) * 16) : kOobOffset;
  }
  return op;
}

// A kW-wide K-major operand: K-row 0 of the tile at `base` (its first column), rows `ld` elements
// apart, `bytes` readable bytes from base on, and `cols` columns from base on that exist (the
// lanes whose chunk lies at or past them load from kOobOffset: zeros, and no address past a
// row's existing columns).
template <int kW = 256>
__device__ __forceinline__ Operand kmajor_operand(const uint16_t* base, int64_t ld, uint64_t bytes, int cols) {
  Operand op;
  op.base = base;
  op.ld = ld;
  op.bytes = bytes;
  op.qstride = (uint32_t)(4 * ld);      // two K-rows (kW = 256)
  const int j = threadIdx.x & 63, w = threadIdx.x >> 6;
#pragma unroll
  for (int q = 0; q < (kW == 256 ? 2 : 4); ++q) {
    int p = w * 256 + q * 64 + j;                       // 16-byte unit of the region
    p = p < kW * 8 ? p : kW * 8 - 1;                    // (waves that do not load this operand)
    const int k = p / (kW / 8), pos = p % (kW / 8);
    const int c = kchunk<kW>(k, pos);
    // kW = 256: the K-rows 4 further (q = 2, 3) have the same chunk (same bits 0-1 and 3 of k)
    op.off[q] = c * 8 < cols ? (uint32_t)((int64_t)k * ld * 2 + (c << 4)) : kOobOffset;
  }
  return op;
}

// ---------------------------------------------------------------------------------------------
// K1: valid-row compaction: the LCE objective drops ignored targets before the projection
// (Sec. 4.2), so no MFMA work is spent on their rows.
// idx[0..Nv) = ascending rows whose target is in [0, V); pos[n] = its index there or -1.
// One workgroup of 16 waves walks the rows in rounds of 1024 consecutive rows (coalesced target
// loads, up to 16 rounds loaded ahead): a row's index is the valid rows of earlier rounds, of
// earlier waves of its round (wave ballots summed through LDS) and of lower lanes of its wave
// (popcount of its ballot), so idx comes out sorted.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void k_compact(const void* targets, int tbytes, int64_t n, int64_t v,
                                                  int ignore, int* idx, int* pos, int* nv_ws,
                                                  int* nv_user, int* status, float* lse_zero,
                                                  float* loss_zero) {
  constexpr int kAhead = 16;
  __shared__ int wsum[2][16];
  __shared__ int bad_any;
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  if (t == 0) bad_any = 0;
  __syncthreads();
  int base = 0, bad = 0;
  for (int64_t g0 = 0; g0 < n; g0 += (int64_t)1024 * kAhead) {
    int64_t tg[kAhead];
#pragma unroll
    for (int r = 0; r < kAhead; ++r) {
      const int64_t i = g0 + (int64_t)r * 1024 + t;
      tg[r] = i < n ? load_target(targets, tbytes, i) : (int64_t)ignore;
    }
#pragma unroll
    for (int r = 0; r < kAhead; ++r) {
      const int64_t i = g0 + (int64_t)r * 1024 + t;
      if (g0 + (int64_t)r * 1024 >= n) break;   // uniform
      const bool ign = tg[r] == (int64_t)ignore;
      const bool ok = i < n && !ign && tg[r] >= 0 && tg[r] < v;
      bad |= (i < n && !ign && !ok);
      const unsigned long long m = __ballot(ok);
      const int below = __popcll(m & ((1ull << lane) - 1ull));
      if (lane == 0) wsum[r & 1][w] = __popcll(m);
      __syncthreads();   // (the buffer written here was last read two rounds ago, before a barrier)
      int before = base, total = 0;
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const int c = wsum[r & 1][k];
        before += k < w ? c : 0;
        total += c;
      }
      if (i < n) {
        if (ok) {
          const int o = before + below;
          idx[o] = (int)i;
          pos[i] = o;
        } else {
          pos[i] = -1;
          if (lse_zero) lse_zero[i] = 0.0f;
          if (loss_zero) loss_zero[i] = 0.0f;
        }
      }
      base += total;
    }
  }
  if (bad) bad_any = 1;  // benign same-value race
  __syncthreads();
  if (t == 0) {
    *nv_ws = base;
    if (nv_user) *nv_user = base;
    if (status) *status = bad_any ? LCE_STATUS_TARGET_OUT_OF_RANGE : 0;
  }
}

// ---------------------------------------------------------------------------------------------
// K2: forward statistics. The objective (Sec. 4.2) needs each valid row's log-sum-exp over the
// whole vocabulary; here it is accumulated tile by tile from logits that are never stored (this
// library's design: the paper states the objective, not an algorithm for it). Two forms, both
// writing per-token partial pairs (max, sum of exp) in log2 units, part[row * npad + token],
// merged by K3:
//  - k_fwd_tile (12 waves, D % 64 == 0): one 384-id x 256-token tile per workgroup, H given as the
//    gathered valid rows Hv; one partial row per vocabulary tile.
//  - k_fwd_stats (8 waves, any D): workgroup (token tile nt, vocabulary partition p) walks the
//    partition's 256-wide tiles with a running pair per token and lane, H's valid rows gathered
//    through idx by the main loop; two partial rows (one per wave row) per partition.
// In both, a tile's S^T = W_tile H^T runs a token's logits down a lane's registers.
// ---------------------------------------------------------------------------------------------
// Tiles are taken in the order of xcd_tile (below), in groups of gw vocabulary tiles (the slab
// rule's width, within the MALL cap, a multiple of 8) by all token tiles, ids fastest: the group's
// W rows stay in the MALL while the token tiles pass, and the workgroups resident on one XCD share
// their W and H tiles through its L2 as in the backward's G launches. One launch covers vt_launch tiles from tm0
// on and writes one partial row per tile (row tm - tm0). When the rows of all tiles would take
// more than 2 D bytes per token (one bf16 row of H), the host launches one group at a time
// instead: group g writes to one of two row sets (by the parity of g), and in launch g >= 1 the
// workgroup of the group's first tile of each token tile first folds the other set (group g - 1,
// complete since launches on a stream run in order) into a running pair per token. The workspace
// thus stays independent of V.
__device__ __forceinline__ void merge_pair(float& m, float& s, float m2, float s2) {
  const float mn = fmaxf(m, m2);
  if (mn == -INFINITY) return;
  s = (m == -INFINITY ? 0.f : s * exp2f(m - mn)) + (m2 == -INFINITY ? 0.f : s2 * exp2f(m2 - mn));
  m = mn;
}

// XCD-aware order of the tiles of a forward or G launch: `tiles` vocabulary tiles by nt token tiles,
// workgroups dealt round-robin to the 8 XCDs (block b runs on XCD b mod 8). The first a = tiles & ~7
// vocabulary tiles go in groups of gw tiles (a and gw multiples of 8; a last group may be narrower)
// by all token tiles, vocabulary tiles fastest: XCD x then takes the tiles = x (mod 8) of each
// group, and a round of its ~32 workgroups shares a few W tiles and a few H tiles, while the group's
// W rows stay in the MALL as the token tiles pass. The last tiles - a (< 8) vocabulary tiles are
// dealt by token tile instead: XCD x takes the token tiles = x (mod 8), each with all of them.
// (Dealt the first way, a group whose width is not a multiple of 8 would give every XCD most of the
// group's W tiles.) False for blocks past the last tile.
__device__ __forceinline__ bool xcd_tile(int b, int tiles, int gw, int nt, int& tm, int& tn) {
  const int a = tiles & ~7, ba = a * nt;
  if (b < ba) {
    const int full = a / gw, g = b / (gw * nt);
    const int wl = g < full ? gw : a - full * gw, r = b - g * gw * nt;
    tm = g * gw + r % wl;
    tn = r / wl;
    return true;
  }
  const int rem = tiles - a, r = b - ba, k = r >> 3;
  if (rem == 0) return false;
  tm = a + k % rem;
  tn = (r & 7) + 8 * (k / rem);
  return tn < nt;
}

__global__ __launch_bounds__(Geo<3>::NT, 3) void k_fwd_tile(const uint16_t* __restrict__ W, int64_t ldw, int v,
                                                            const uint16_t* __restrict__ Hv, int64_t ldh,
                                                            const int* __restrict__ nv_ptr, int d, int tm0,
                                                            int vt_launch, int gw, int nt_max,
                                                            float* __restrict__ part_m, float* __restrict__ part_s,
                                                            const float* __restrict__ prev_m,
                                                            const float* __restrict__ prev_s, int wprev,
                                                            float* __restrict__ run_m, float* __restrict__ run_s,
                                                            int run_init, int npad, float scale2) {
  constexpr int WM = 3, TM = Geo<WM>::TM;
  __shared__ __attribute__((aligned(16))) char smem[Geo<WM>::LDS];
  int tl, tn;   // launch-relative vocabulary tile, token tile
  if (!xcd_tile((int)blockIdx.x, vt_launch, gw, nt_max, tl, tn)) return;
  const int tm = tm0 + tl;
  const int nv = *nv_ptr;
  const int n0 = tn * TILE;
  if (n0 >= nv) return;
  const int v0 = tm * TM, vleft = v - v0;
  if (prev_m && tl == 0 && threadIdx.x < TILE) {
    const int tok = n0 + threadIdx.x;
    if (tok < nv) {
      float m = -INFINITY, s = 0.f;
      if (!run_init) {
        m = run_m[tok];
        s = run_s[tok];
      }
#pragma unroll 8
      for (int q = 0; q < wprev; ++q) merge_pair(m, s, prev_m[(int64_t)q * npad + tok], prev_s[(int64_t)q * npad + tok]);
      run_m[tok] = m;
      run_s[tok] = s;
    }
  }
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, wr = wave >> 2, wc = wave & 3;

  const Operand opb = dense_operand(Hv + (int64_t)n0 * ldh, nv - n0, ldh);
  f32x16_t acc[4][2];
  // d % 64 == 0 (host); the last vocabulary tile may hold fewer than TM rows of W
  if (vleft >= TM)
    mma_mainloop<1, OP_DENSE, OP_DENSE, WM, false>(acc, dense_operand(W + (int64_t)v0 * ldw, vleft, ldw), opb, d,
                                                   smem);
  else
    mma_mainloop<1, OP_GATHER, OP_DENSE, WM, false>(acc, masked_dense_operand<TM>(W + (int64_t)v0 * ldw, vleft, ldw),
                                                    opb, d, smem);
  // the main loop ends with a barrier: its LDS is free for the wave rows' pairs [3][256] (m, s)
  float* red_m = reinterpret_cast<float*>(smem);
  float* red_s = red_m + WM * TILE;

  // rows (vocabulary ids) of this lane: v0 + wr*128 + 32 bi + 8 (r/4) + 4 (lane/32) + r%4
  const int vb = wr * 128 + (lane >> 5) * 4;
  // the rows past V of the last vocabulary tile drop out of the max and the sum; every other tile
  // takes a path with no per-element test (a runtime test would be kept, as masks, on every tile)
  auto mask_rows = [&](auto kRagged) {
    if constexpr (decltype(kRagged)::value) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
#pragma unroll
          for (int r = 0; r < 16; ++r)
            if (vb + i * 32 + (r >> 2) * 8 + (r & 3) >= vleft) acc[i][j][r] = -INFINITY;
    }
  };
  if (vleft < TM) mask_rows(std::true_type{});
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, acc[i][j][r]);
    const float nm = mx * scale2;
    float st = 0.f;
    if (nm != -INFINITY) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) st += __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], scale2, -nm));
    }
    // merge the two lane halves (disjoint ids of the same tokens)
    const float om = __shfl_xor(nm, 32), os = __shfl_xor(st, 32);
    const float mm = fmaxf(nm, om);
    float sm = 0.f;
    if (mm != -INFINITY) {
      sm = (nm == -INFINITY ? 0.f : st * __builtin_amdgcn_exp2f(nm - mm)) +
           (om == -INFINITY ? 0.f : os * __builtin_amdgcn_exp2f(om - mm));
    }
    if (lane < 32) {
      const int t = wr * TILE + wc * 64 + j * 32 + lane;
      red_m[t] = mm;
      red_s[t] = sm;
    }
  }
  __syncthreads();
  // merge the three wave rows in order; one thread per token of the tile
  if (threadIdx.x < TILE) {
    const int t = threadIdx.x, tok = n0 + t;
    float m = red_m[t], s = red_s[t];
#pragma unroll
    for (int q = 1; q < WM; ++q) {
      const float m2 = red_m[q * TILE + t], s2 = red_s[q * TILE + t];
      const float mn = fmaxf(m, m2);
      if (mn != -INFINITY)
        s = (m == -INFINITY ? 0.f : s * __builtin_amdgcn_exp2f(m - mn)) +
            (m2 == -INFINITY ? 0.f : s2 * __builtin_amdgcn_exp2f(m2 - mn));
      m = mn;
    }
    if (tok < nv) {
      part_m[(int64_t)tl * npad + tok] = m;
      part_s[(int64_t)tl * npad + tok] = s;
    }
  }
}

template <int WM>
__global__ __launch_bounds__(Geo<WM>::NT, WM) void k_fwd_stats(const uint16_t* __restrict__ W, int64_t ldw, int v,
                                                           const uint16_t* __restrict__ H, int64_t ldh, int64_t n,
                                                           const int* __restrict__ idx, const int* __restrict__ nv_ptr,
                                                           int d, int nparts, int nt_max, int vt_count,
                                                           float* __restrict__ part_m, float* __restrict__ part_s,
                                                           int npad, float scale2) {
  // scale2 = log2(e) / T: partials are kept in base-2 units of the logits divided by T.
  static_assert(WM == 2, "");
  constexpr int TM = Geo<WM>::TM;
  __shared__ __attribute__((aligned(16))) char smem[Geo<WM>::LDS];
  // Workgroups are dispatched round-robin over the 8 XCDs (block b runs on XCD b % 8). Each XCD
  // owns whole vocabulary partitions (p = xcd + 8 k, k < ppx) and runs its workgroups in rounds of
  // about 32 (one per CU): every round covers all ppx partitions for a group of 32 / ppx token
  // tiles, so the resident workgroups share ppx W tiles and 32 / ppx H tiles through the XCD's L2
  // (12 distinct tiles per 32 workgroups at ppx = 4, where one partition over 32 token tiles
  // would stream 32 distinct H tiles). The last round takes the token tiles that are left.
  int nt, p;
  if (nparts % 8 == 0) {
    const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
    const int ppx = nparts >> 3;
    const int gn = ppx >= 32 ? 1 : 32 / ppx;
    const int r = slot / (ppx * gn), rem = slot % (ppx * gn);
    p = xcd + 8 * (rem % ppx);
    nt = r * gn + rem / ppx;
  } else {
    nt = blockIdx.x % nt_max;
    p = blockIdx.x / nt_max;
  }
  const int nv = *nv_ptr;
  const int n0 = nt * TILE;
  if (n0 >= nv) return;
  const int vt0 = (int)((int64_t)p * vt_count / nparts), vt1 = (int)((int64_t)(p + 1) * vt_count / nparts);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, wr = wave >> 2, wc = wave & 3;
  const Operand opb = gather_operand(H, n, ldh, idx, n0, nv);

  f32x16_t acc[4][2];
  float m2[2], ss[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) { m2[j] = -INFINITY; ss[j] = 0.f; }

  for (int vt = vt0; vt < vt1; ++vt) {
    const int v0 = vt * TM;
    const int vleft = v - v0;
    if (vleft >= TM)
      mma_mainloop<2, OP_DENSE, OP_GATHER, WM>(acc, dense_operand(W + (int64_t)v0 * ldw, vleft, ldw), opb, d, smem);
    else
      mma_mainloop<2, OP_GATHER, OP_GATHER, WM>(acc, masked_dense_operand<TM>(W + (int64_t)v0 * ldw, vleft, ldw), opb,
                                                d, smem);

    // rows (vocabulary ids) of this lane: v0 + wr*128 + 32 bi + 8 (r/4) + 4 (lane/32) + r%4
    const int vb = wr * 128 + (lane >> 5) * 4;
    const bool ragged = vleft < TM;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          if (ragged && (vb + i * 32 + (r >> 2) * 8 + (r & 3)) >= vleft) acc[i][j][r] = -INFINITY;
          mx = fmaxf(mx, acc[i][j][r]);
        }
      const float nm = fmaxf(m2[j], mx * scale2);
      if (nm == -INFINITY) continue;
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], scale2, -nm));
      ss[j] = (m2[j] == -INFINITY ? 0.f : ss[j] * __builtin_amdgcn_exp2f(m2[j] - nm)) + s;
      m2[j] = nm;
    }
  }
  // merge the two lane halves (disjoint vocabulary rows), then write this wave row's partial
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const float om = __shfl_xor(m2[j], 32), os = __shfl_xor(ss[j], 32);
    const float nm = fmaxf(m2[j], om);
    float s = 0.f;
    if (nm != -INFINITY) {
      s = (m2[j] == -INFINITY ? 0.f : ss[j] * __builtin_amdgcn_exp2f(m2[j] - nm)) +
          (om == -INFINITY ? 0.f : os * __builtin_amdgcn_exp2f(om - nm));
    }
    const int tok = n0 + wc * 64 + j * 32 + (lane & 31);
    if (lane < 32 && tok < nv) {
      const int64_t o = (int64_t)(WM * p + wr) * npad + tok;
      part_m[o] = nm;
      part_s[o] = s;
    }
  }
}

// ---------------------------------------------------------------------------------------------
// K3: per valid token: merge the vocabulary partials into lse, take the target logit
// s[n, t_n] = H[n] . W[t_n] in fp32, and the per-row loss l_n = lse_n - s[n, t_n].
// A workgroup of 16 waves serves 64 consecutive tokens. First each wave folds every 16th partial
// row (rows w, w + 16, ...) for the 64 tokens, one token per lane (reads coalesced along the
// tokens), and the 16 results are merged in wave order; then each wave takes the target logits of
// 4 tokens, one wave-wide dot product each. All reductions run in a fixed order.
// ---------------------------------------------------------------------------------------------
constexpr int kCombTok = 64;

__global__ __launch_bounds__(1024) void k_combine(const uint16_t* __restrict__ H, int64_t ldh,
                                                  const uint16_t* __restrict__ W, int64_t ldw,
                                                  const void* targets, int tbytes, int64_t id0, int64_t v_local,
                                                  const int* __restrict__ idx, const int* __restrict__ nv_ptr,
                                                  int d, int nparts2, const float* __restrict__ part_m,
                                                  const float* __restrict__ part_s, int npad,
                                                  const float* __restrict__ run_m, const float* __restrict__ run_s,
                                                  float* __restrict__ lse_out, float* __restrict__ terms,
                                                  float* __restrict__ per_token, float* __restrict__ tgt_part) {
  // run_m / run_s (may be null): a running pair per token folded in before the partial rows
  __shared__ float red_m[16][kCombTok], red_s[16][kCombTok], lse_t[kCombTok];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int i0 = blockIdx.x * kCombTok;
  const int nv = *nv_ptr;
  if (i0 >= nv) return;
  {
    const int i = i0 + lane;
    float m = -INFINITY, s = 0.f;
    if (i < nv && wave == 0 && run_m) {
      m = run_m[i];
      s = run_s[i];
    }
    if (i < nv)
      for (int q = wave; q < nparts2; q += 16) merge_pair(m, s, part_m[(int64_t)q * npad + i], part_s[(int64_t)q * npad + i]);
    red_m[wave][lane] = m;
    red_s[wave][lane] = s;
  }
  __syncthreads();
  if (wave == 0) {
    float m = red_m[0][lane], s = red_s[0][lane];
    for (int q = 1; q < 16; ++q) merge_pair(m, s, red_m[q][lane], red_s[q][lane]);
    lse_t[lane] = (m + log2f(s)) * kLn2;
  }
  __syncthreads();
  for (int t = 0; t < kCombTok / 16; ++t) {
    const int li = wave * (kCombTok / 16) + t, i = i0 + li;
    if (i >= nv) break;
    const int row = idx[i];
    // target id relative to this W's first row (id0 > 0 only for a vocabulary shard, which may
    // not hold the target: then its target logit is 0)
    const int64_t tl = load_target(targets, tbytes, row) - id0;
    float dot = 0.f;
    if (tl >= 0 && tl < v_local) {
      const uint4* hr = reinterpret_cast<const uint4*>(H + (int64_t)row * ldh);
      const uint4* wt = reinterpret_cast<const uint4*>(W + tl * ldw);
      for (int c = lane; c < d / 8; c += 64) {
        const uint4 a = hr[c], b = wt[c];
        const uint32_t av[4] = {a.x, a.y, a.z, a.w}, bv[4] = {b.x, b.y, b.z, b.w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          dot = fmaf(bf16_to_f32(av[q] & 0xFFFF), bf16_to_f32(bv[q] & 0xFFFF), dot);
          dot = fmaf(bf16_to_f32(av[q] >> 16), bf16_to_f32(bv[q] >> 16), dot);
        }
      }
      dot = wave_sum(dot);
    }
    if (lane == 0) {
      const float lse = lse_t[li];
      lse_out[row] = lse;
      if (tgt_part) {
        tgt_part[row] = dot;
      } else {
        terms[i] = lse - dot;
        if (per_token) per_token[row] = lse - dot;
      }
    }
  }
}

// Combine of vocabulary shards: lse = log sum_g exp(lse_g) (max-shifted, shards in order) and the
// target logit sum_g tgt_g (one shard holds it), per valid token; one thread per token.
__global__ __launch_bounds__(256) void k_shard_combine(int g_count, const float* __restrict__ lse_parts,
                                                       const float* __restrict__ tgt_parts, int64_t ld,
                                                       const int* __restrict__ idx, const int* __restrict__ nv_ptr,
                                                       float* __restrict__ lse_out, float* __restrict__ terms,
                                                       float* __restrict__ per_token) {
  const int i = blockIdx.x * 256 + threadIdx.x;
  if (i >= *nv_ptr) return;
  const int row = idx[i];
  float mm = -INFINITY;
  for (int g = 0; g < g_count; ++g) mm = fmaxf(mm, lse_parts[g * ld + row]);
  float se = 0.f, z = 0.f;
  for (int g = 0; g < g_count; ++g) {
    se += exp2f((lse_parts[g * ld + row] - mm) * kLog2e);
    z += tgt_parts[g * ld + row];
  }
  const float lse = mm + log2f(se) * kLn2;
  lse_out[row] = lse;
  terms[i] = lse - z;
  if (per_token) per_token[row] = lse - z;
}

// K3b: loss = sum or mean of the per-row terms, fixed-order fp64 tree.
__global__ __launch_bounds__(1024) void k_loss(const float* __restrict__ terms, const int* __restrict__ nv_ptr,
                                               int reduction, float* __restrict__ loss) {
  __shared__ double red[1024];
  const int t = threadIdx.x;
  const int nv = *nv_ptr;
  double s = 0.0;
  for (int i = t; i < nv; i += 1024) s += (double)terms[i];
  red[t] = s;
  __syncthreads();
  for (int w = 512; w > 0; w >>= 1) {
    if (t < w) red[t] += red[t + w];
    __syncthreads();
  }
  if (t == 0) {
    double r = red[0];
    if (nv == 0) r = 0.0;
    else if (reduction == LCE_REDUCE_MEAN) r /= (double)nv;
    *loss = (float)r;
  }
}

__global__ void k_fwd_empty(float* loss, int* nv_user, int* status) {
  if (threadIdx.x == 0) {
    if (loss) *loss = 0.f;
    *nv_user = 0;
    if (status) *status = 0;
  }
}

// ---------------------------------------------------------------------------------------------
// Hv[i][:] = H[idx[i]][:] for i < Nv (rows of d elements), zero rows up to round_up(Nv, 64): the
// valid rows of H made contiguous. It is the B operand of the backward G tiles (row-major) and of
// the dW contraction (K-major over tokens), so neither main loop gathers rows itself.
// ---------------------------------------------------------------------------------------------
__global__ __launch_bounds__(256) void k_gather_rows(const uint16_t* __restrict__ H, int64_t ldh,
                                                     const int* __restrict__ idx, const int* __restrict__ nv_ptr,
                                                     int d, uint16_t* __restrict__ Hv) {
  const int nv = *nv_ptr;
  const int64_t rows = (nv + 63) / 64 * 64;
  const int cpr = d / 8;   // 16-byte chunks per row
  const int64_t total = rows * cpr;
  for (int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int64_t i = e / cpr;
    const int c = (int)(e - i * cpr);
    uint4 v = make_uint4(0, 0, 0, 0);
    if (i < nv) v = *reinterpret_cast<const uint4*>(H + (int64_t)idx[i] * ldh + c * 8);
    *reinterpret_cast<uint4*>(Hv + i * d + c * 8) = v;
  }
}

// Tile scheduling of the dH launches whose K the host splits into parts (launches with fewer
// tiles than CUs; one copy of this grid per part). Workgroups are dispatched round-robin over the
// 8 XCDs (block b runs on XCD b % 8), each with its own L2. XCD x owns the band of row tiles
// [x T / 8, (x + 1) T / 8) (T = live row tiles) and walks it column by column, so the workgroups
// resident on one XCD share the band's A tiles and a few B tiles in its L2, and each A operand is
// fetched by one XCD only. The grid is 8 * ceil(T_max / 8) * tn_count blocks; blocks past the live
// tiles return false.
__device__ __forceinline__ bool band_tile(int blk, int tm_live, int tn_count, int& tm, int& tn) {
  const int x = blk & 7, k = blk >> 3;
  const int r0 = (x * tm_live) >> 3, r1 = ((x + 1) * tm_live) >> 3;
  const int rows = r1 - r0;
  if (rows <= 0 || k >= rows * tn_count) return false;
  tm = r0 + k % rows;
  tn = k / rows;
  return true;
}

// dH launches whose K the host did not split. With T = tm_live x dt live output tiles (tm_live =
// ceil(Nv / 384) row tiles of 384 tokens, dt column tiles of 256), XCD x takes the tiles [c0(x),
// c0(x + 1)) of a balanced cut, c0(x) = floor(x T / 8), in an order that keeps consecutive tiles on
// few operand tiles: bands of 4 row tiles, each walked column by column. An XCD runs its ~32
// resident workgroups in rounds; the n_tail tiles of its last, partial round are split along K
// into dh_tail_parts(n_tail) parts, so that they fill that round instead of leaving most of its
// CUs idle. Part 0 of a tile accumulates into the tile's rows of the accumulator (row stride D);
// part z >= 1 of tail tile t into slot dh_slot0(x) + (z - 1) * n_tail + t, a 384 x 256 fp32 block
// (row stride 256) in the accumulator's rows at or past tm_live * 384, which hold no valid token.
// When those rows cannot hold every slot, no tile is split. The finalise adds the parts in order.
constexpr int kDhBand = 4;                       // row tiles per band
constexpr int64_t kDhSlot = 384 * 256;           // floats per slot
__device__ __forceinline__ int dh_c0(int x, int t) { return (int)(((int64_t)x * t) >> 3); }
__device__ __forceinline__ int dh_tail_parts(int n_tail) {
  return n_tail > 0 && n_tail <= 16 ? (32 / n_tail < 8 ? 32 / n_tail : 8) : 1;
}
// slots taken by the XCDs before x (the slots are numbered XCD by XCD, each XCD's in part-major
// order); dh_slot0(8, t) is the total
__device__ __forceinline__ int dh_slot0(int x, int t) {
  int n = 0;
  for (int y = 0; y < x; ++y) {
    const int nt = (dh_c0(y + 1, t) - dh_c0(y, t)) & 31;
    n += (dh_tail_parts(nt) - 1) * nt;
  }
  return n;
}
__device__ __forceinline__ bool dh_tail_fits(int t, int tm_live, int d, int acc_rows) {
  return (int64_t)dh_slot0(8, t) * kDhSlot <= (int64_t)(acc_rows - tm_live * 384) * d;
}
__device__ __forceinline__ void dh_band_tile(int l, int tm_live, int dt, int& tm, int& tn) {
  const int band = l / (kDhBand * dt), r0 = band * kDhBand;
  const int rows = tm_live - r0 < kDhBand ? tm_live - r0 : kDhBand;
  const int k = l - band * kDhBand * dt;
  tm = r0 + k % rows;
  tn = k / rows;
}
__device__ __forceinline__ int dh_band_index(int tm, int tn, int tm_live, int dt) {
  const int band = tm / kDhBand, r0 = band * kDhBand;
  const int rows = tm_live - r0 < kDhBand ? tm_live - r0 : kDhBand;
  return band * kDhBand * dt + tn * rows + (tm - r0);
}

// scale c = g / n_norm (mean) or g (sum), 0 when the count is 0; for NONE the caller reads
// the per-token gradient instead
__device__ __forceinline__ float grad_scale(const float* grad, const int* n_norm, int reduction) {
  if (reduction == LCE_REDUCE_NONE) return 0.f;
  const float g = *grad;
  if (reduction == LCE_REDUCE_SUM) return g;
  const int nn = *n_norm;
  return nn > 0 ? g / (float)nn : 0.f;
}

// ---------------------------------------------------------------------------------------------
// K4: softmax-gradient tile for one vocabulary slab. Tile (vocabulary tile tm, token tile tn) of
// S^T = W_slab Hv^T is recomputed and turned into G = c (exp(s - lse) - onehot), rounded to
// bf16 and written as G[token][v] (row stride vc). Every tile is written whole: entries of tokens
// at or beyond Nv and of ids at or beyond the slab width are zeros, so the two contractions that
// read G (dH with K = ids, dW with K = tokens, G read K-major) need no masking of G.
// ---------------------------------------------------------------------------------------------
// The same kernel serves the distillation loss (KD) with soft targets, in four modes:
//   G_ONEHOT  LCE: G = c (softmax - onehot(t))
//   G_SOFT    KD student: G = c (softmax(z/T) - P) / T, P the teacher's probabilities of this slab
//   Q_SOFT    KD student forward: per token, sum over the tile's ids of P * z / T (partials qpart)
//   P_WRITE   KD teacher: P = softmax(z/T) of this slab, fp32, P[v][token] (row stride ldt)
//   G_SOFT_Q  KD student, forward and backward in one pass: G_SOFT and Q_SOFT together
// scale2 = log2(e) / T (log2(e) for LCE), inv_t = 1 / T; lse is that of the scaled logits.
enum GMode { G_ONEHOT = 0, G_SOFT = 1, Q_SOFT = 2, P_WRITE = 3, G_SOFT_Q = 4 };

template <int kMode, int WM>
__global__ __launch_bounds__(Geo<WM>::NT, WM) void k_bwd_g(const uint16_t* __restrict__ W, int64_t ldw, int64_t v0, int vs,
                                                       const uint16_t* __restrict__ H, int64_t ldh, int64_t n,
                                                       const void* targets, int tbytes, int64_t id0,
                                                       const int* __restrict__ idx, const int* __restrict__ nv_ptr,
                                                       const float* __restrict__ lse, const float* __restrict__ grad,
                                                       const int* __restrict__ n_norm, int reduction, int d, int tm_count,
                                                       uint16_t* __restrict__ G, int vc, int ldt,
                                                       float scale2, float inv_t, float* __restrict__ P,
                                                       float* __restrict__ qpart, int64_t qrow, int gsub) {
  // 12 waves (WM = 3, 384 ids per tile) serve the one-hot LCE gradient when D % 64 == 0; the
  // distillation modes and other widths keep 8 waves and the LDS-staged epilogue below
  static_assert(WM == 2 || kMode == G_ONEHOT || kMode == P_WRITE, "");
  constexpr int TM = Geo<WM>::TM;
  __shared__ __attribute__((aligned(16))) char smem[Geo<WM>::LDS];
  const int nv = *nv_ptr;
  // tiles in the XCD-aware order of xcd_tile, in groups of gsub id tiles (ldt = Npad: ldt / 256
  // token tiles)
  int tm, tn;
  if (!xcd_tile((int)blockIdx.x, tm_count, gsub, ldt / TILE, tm, tn)) return;
  const int n0 = tn * TILE;
  if (n0 >= nv) return;
  const int vt0 = tm * TM;                   // slab-relative
  const int vleft = vs - vt0;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, wr = wave >> 2, wc = wave & 3;

  const uint16_t* wt = W + (v0 + vt0) * ldw;
  f32x16_t acc[4][2];
  // the last tile of the vocabulary may hold fewer than TM rows of W
  if constexpr (WM == 3) {
    // H is the gathered valid rows Hv (row stride ldh = d): a dense operand; d % 64 == 0 (host)
    const Operand opb = dense_operand(H + (int64_t)n0 * ldh, nv - n0, ldh);
    if (vleft >= TM)
      mma_mainloop<1, OP_DENSE, OP_DENSE, WM, false>(acc, dense_operand(wt, vleft, ldw), opb, d, smem);
    else
      mma_mainloop<1, OP_GATHER, OP_DENSE, WM, false>(acc, masked_dense_operand<TM>(wt, vleft, ldw), opb, d, smem);
  } else {
    const Operand opb = gather_operand(H, n, ldh, idx, n0, nv);
    if (vleft >= TM)
      mma_mainloop<2, OP_DENSE, OP_GATHER, WM>(acc, dense_operand(wt, vleft, ldw), opb, d, smem);
    else
      mma_mainloop<2, OP_GATHER, OP_GATHER, WM>(acc, masked_dense_operand<TM>(wt, vleft, ldw), opb, d, smem);
  }

  // the gradient scale exists only for the modes that write G (the probability and Q passes get
  // no upstream gradient: grad and n_norm may be null there)
  constexpr bool kWritesG = kMode == G_ONEHOT || kMode == G_SOFT || kMode == G_SOFT_Q;
  const float c_all = kWritesG ? grad_scale(grad, n_norm, reduction) : 0.f;
  int tok[2], tgt[2];
  float l2[2], cj[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    tok[j] = n0 + wc * 64 + j * 32 + (lane & 31);
    if (tok[j] < nv) {
      const int row = idx[tok[j]];
      l2[j] = lse[row] * kLog2e;
      tgt[j] = kMode == G_ONEHOT ? (int)(load_target(targets, tbytes, row) - id0 - v0) - vt0 : -1;
      cj[j] = kWritesG && reduction == LCE_REDUCE_NONE ? grad[row] : c_all;
    } else {
      l2[j] = 0.f;
      tgt[j] = -1;
      cj[j] = 0.f;
    }
  }
  const int vb = wr * 128 + (lane >> 5) * 4;  // tile-relative vocabulary row base of this lane
  if constexpr (WM == 3 && kMode == G_ONEHOT) {
    // G straight from registers. A lane holds 4 consecutive ids of a token row per (block, group
    // of 8 ids), the other 4 sit in lane L ^ 32; one lane swap across the wave halves
    // (permlane32 swap) per pair of groups gives each lane 8 consecutive ids (lanes < 32 the even
    // group, the others the odd one), stored as 16 bytes. Rows of tokens >= Nv and ids >= the
    // slab width get zeros, so the whole 256 x 384 tile is written (the slab width vc is a
    // multiple of 384).
    const i32x4_t rg = make_rsrc_words(G + (int64_t)n0 * vc, (uint64_t)TILE * vc * 2);
    const uint32_t voff = (uint32_t)(((wc * 64 + (lane & 31)) * vc + vt0 + wr * 128 + (lane >> 5) * 8) * 2);
    // A tile whose tokens are all valid and whose ids all lie in the slab needs no test per
    // element; on the other tiles the values out of range are replaced by zeros (a select, not a
    // branch per element: the exponential of a row past Nv may be anything, even NaN).
    auto store_tile = [&](auto kFull) {
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        const bool tok_ok = tok[j] < nv;
        // the lane's element (i, q, e) is the target's when dt == 32 i + 8 q + e: one compare
        // with a constant per element, and the one-hot term folded into the scaling fma
        const int dt = tgt[j] - vb;
        const float nc = -cj[j];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
          for (int p = 0; p < 2; ++p) {
            u32x2_t pk[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
              const int q = 2 * p + h;
              float gq[4];
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                const int k = i * 32 + q * 8 + e;
                const float ex = __builtin_amdgcn_exp2f(fmaf(acc[i][j][q * 4 + e], scale2, -l2[j]));
                float g = fmaf(cj[j], ex, dt == k ? nc : 0.f);
                if constexpr (!decltype(kFull)::value) g = (tok_ok && vb + k < vleft) ? g : 0.f;
                gq[e] = g;
              }
              pk[h].x = pack_bf16x2(gq[0], gq[1]);
              pk[h].y = pack_bf16x2(gq[2], gq[3]);
            }
            // lane L < 32: (its group 2p ids 0-3, lane L + 32's ids 4-7); lane L + 32: (lane L's
            // group 2p + 1 ids 0-3, its own ids 4-7)
            const auto sx = __builtin_amdgcn_permlane32_swap(pk[0].x, pk[1].x, false, false);
            const auto sy = __builtin_amdgcn_permlane32_swap(pk[0].y, pk[1].y, false, false);
            const i32x4_t v16 = {(int)sx[0], (int)sy[0], (int)sx[1], (int)sy[1]};
            const uint32_t so = (uint32_t)((j * 32 * vc + i * 32 + p * 16) * 2);
            // (the compiled code may rewrite v16's registers right after the store: padded)
            buffer_store16_padded(v16, rg, voff, so);
          }
      }
    };
    if (n0 + TILE <= nv && vleft >= TM) store_tile(std::true_type{});
    else store_tile(std::false_type{});
    return;
  } else if constexpr (kMode == P_WRITE || kMode == Q_SOFT) {
    // P[v][token] rows of this tile: lanes of a half-wave hold 32 consecutive tokens of one row
    float q[2] = {0.f, 0.f};
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      if (tok[j] >= nv) continue;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        if constexpr (kMode == P_WRITE) {
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int vr = vb + i * 32 + (r >> 2) * 8 + (r & 3);
            if (vr < vleft)
              P[(int64_t)(vt0 + vr) * ldt + tok[j]] = __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], scale2, -l2[j]));
          }
        } else {
          // the block's 16 probabilities are loaded together, then used
          float pt[16];
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int vr = vb + i * 32 + (r >> 2) * 8 + (r & 3);
            pt[r] = vr < vleft ? P[(int64_t)(vt0 + vr) * ldt + tok[j]] : 0.f;
          }
#pragma unroll
          for (int r = 0; r < 16; ++r) q[j] = fmaf(pt[r], acc[i][j][r] * inv_t, q[j]);
        }
      }
    }
    if constexpr (kMode == Q_SOFT) {
      // the two lane halves hold disjoint vocabulary rows of the same tokens
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        q[j] += __shfl_xor(q[j], 32);
        if (lane < 32 && tok[j] < nv) qpart[(qrow + 2 * tm + wr) * ldt + tok[j]] = q[j];
      }
    }
    return;
  }
  // G values in place, then the bf16 tile goes through LDS (free after the main loop) as
  // T[token][v], 512-byte rows whose 16-byte chunk c sits at c ^ (token & 31), so that the
  // token-major rows of G leave with wide coalesced stores. Within a chunk the two 8-byte halves
  // (ids 0-3, 4-7) trade places in token rows with bit 4 set: the 32 lanes of a half-wave, which
  // hold the same half of 32 consecutive token rows, then write 32 distinct 8-byte bank slots.
  char* T = smem;
  float qs[2] = {0.f, 0.f};
  // a tile whose tokens are all valid and whose ids all lie in the slab tests nothing per element
  // (a runtime test would be kept, as masks and branches, on every tile)
  auto fill = [&](auto kFull) {
    constexpr bool kF = decltype(kFull)::value;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const bool tok_ok = kF || tok[j] < nv;
      const int nl = wc * 64 + j * 32 + (lane & 31);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float pt[16];
        if constexpr (kMode == G_SOFT || kMode == G_SOFT_Q) {
          // the block's 16 teacher probabilities are loaded together, then used
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int vr = vb + i * 32 + (r >> 2) * 8 + (r & 3);
            pt[r] = (kF || (tok_ok && vr < vleft)) ? P[(int64_t)(vt0 + vr) * ldt + tok[j]] : 0.f;
          }
        }
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          float gq[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int r = q * 4 + e;
            const int vr = vb + i * 32 + q * 8 + e;
            float g = 0.f;
            if (kF || (tok_ok && vr < vleft)) {
              const float e2 = __builtin_amdgcn_exp2f(fmaf(acc[i][j][r], scale2, -l2[j]));
              if constexpr (kMode == G_SOFT || kMode == G_SOFT_Q) {
                g = cj[j] * inv_t * (e2 - pt[r]);
                if constexpr (kMode == G_SOFT_Q) qs[j] = fmaf(pt[r], acc[i][j][r] * inv_t, qs[j]);
              } else {
                g = cj[j] * e2;
                if (vr == tgt[j]) g -= cj[j];
              }
            }
            gq[e] = g;
          }
          const int vl = vb + i * 32 + q * 8;
          u32x2_t pk;
          pk.x = pack_bf16x2(gq[0], gq[1]);
          pk.y = pack_bf16x2(gq[2], gq[3]);
          const uint32_t a = (uint32_t)(nl * 512 + ((((vl >> 3) ^ (nl & 31))) << 4) +
                                        ((((vl >> 2) & 1) ^ ((nl >> 4) & 1)) << 3));
          *reinterpret_cast<u32x2_t*>(T + a) = pk;
        }
      }
    }
  };
  if (n0 + TILE <= nv && vleft >= TM) fill(std::true_type{});
  else fill(std::false_type{});
  if constexpr (kMode == G_SOFT_Q) {
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      qs[j] += __shfl_xor(qs[j], 32);
      if (lane < 32 && tok[j] < nv) qpart[(qrow + 2 * tm + wr) * ldt + tok[j]] = qs[j];
    }
  }
  __syncthreads();
  // G rows, the whole tile (rows of tokens >= Nv are zeros): 16-byte chunks, one 512-byte row
  // per 32 threads
#pragma unroll 4
  for (int it = 0; it < 16; ++it) {
    const int q = threadIdx.x + NTHREADS * it;
    const int nl = q >> 5, ch = q & 31;
    i32x4_t val = *reinterpret_cast<const i32x4_t*>(T + nl * 512 + ((ch ^ (nl & 31)) << 4));
    if (nl & 16) val = (i32x4_t){val.z, val.w, val.x, val.y};
    store16_padded(G + (int64_t)(n0 + nl) * vc + vt0 + ch * 8, val);
  }
}

// K5: dW[v0 + m][dd] = sum_k G[k][m] Hv[k][dd] over k < round_up(Nv, 64), G [Npad][vc] and the
// gathered valid rows Hv [Npad][D] both read K-major (transposing LDS reads); tiles of (128 WM)
// ids x 256 hidden columns. The epilogue either writes the block in bf16 (each element once), adds it to the bf16
// values already there, or hands each bf16-rounded element straight to the AdamW update of W (the
// in-backward step). Its accesses go through buffer resources over the tile's rows below the slab
// width (rows past it read 0 and drop their stores): a per-lane 32-bit offset and a wave-uniform
// row offset per element, so that the accumulators are nearly the only registers it holds.
enum DwMode { DW_STORE = 0, DW_ACCUMULATE = 1, DW_ADAMW = 2 };

// One dW tile (block blk of the dW grid, smem the workgroup's LDS).
template <int kMode, int WM>
__device__ __forceinline__ void dw_tile(char* smem, int blk, const uint16_t* __restrict__ G, int vc, int ldt, int vs,
                                        const uint16_t* __restrict__ Hv, int d, const int* __restrict__ nv_ptr,
                                        int tm_count, uint16_t* __restrict__ dW, int64_t v0, const AdamWState& st,
                                        const AdamWConst& oc) {
  constexpr int TM = Geo<WM>::TM;
  // the slab's T = tm_count x dt tiles in the balanced cut of the dH launches: XCD x takes
  // [c0(x), c0(x + 1)), walked in bands of 4 row tiles, column by column
  const int dt = (d + TILE - 1) / TILE, t = tm_count * dt, x = blk & 7, k = blk >> 3;
  const int c0 = dh_c0(x, t);
  if (k >= dh_c0(x + 1, t) - c0) return;
  int tm, tn;
  dh_band_tile(c0 + k, tm_count, dt, tm, tn);
  const int m0 = tm * TM, d0 = tn * TILE;
  const int nv = *nv_ptr;
  const int kpad = ((nv + KPAD - 1) / KPAD) * KPAD;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, wr = wave >> 2, wc = wave & 3;
  // ldt = Npad: G has Npad rows of vc ids, Hv Npad rows of d hidden columns
  const Operand opa = kmajor_operand<TM>(G + m0, vc, ((uint64_t)ldt * vc - m0) * 2, vc - m0);
  const Operand opb = kmajor_operand<TILE>(Hv + d0, d, ((uint64_t)ldt * d - d0) * 2, d - d0);
  f32x16_t acc[4][2];
  mma_mainloop<1, OP_KMAJOR, OP_KMAJOR, WM, false>(acc, opa, opb, kpad, smem);

  const int rows = vs - m0 < TM ? vs - m0 : TM;             // valid id rows of this tile
  const int64_t r0 = v0 + m0;                               // its first row of W / dW
  const int dc = d0 + wc * 64 + (lane & 31);
  const int lrow = wr * 128 + (lane >> 5) * 4;              // this lane's first tile row
  const bool col_ok[2] = {dc < d, dc + 32 < d};
  // row offset (in elements of a row of `stride`) of block i, register r
  auto erow = [](int i, int r) { return i * 32 + (r >> 2) * 8 + (r & 3); };
  // on the last tile of the vocabulary, the rows past it are not accessed at all (dW and the
  // optimizer state end there)
  const bool partial = rows < TM;
  auto row_ok = [&](int i, int r) { return !partial || lrow + erow(i, r) < rows; };
  if constexpr (kMode != DW_ADAMW) {
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(dW + r0 * d, (uint64_t)rows * d * 2);
    const uint32_t voff = (uint32_t)((lrow * d + dc) * 2);
    // tiles with all their rows in the vocabulary and all columns inside D test nothing per element
    auto store_tile = [&](auto kFull) {
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          if (!decltype(kFull)::value && !col_ok[j]) continue;
          float old[16];
          if constexpr (kMode == DW_ACCUMULATE) {
#pragma unroll
            for (int r = 0; r < 16; ++r) {
              const uint32_t so = (uint32_t)((erow(i, r) * d + j * 32) * 2);
              old[r] = (decltype(kFull)::value || row_ok(i, r))
                           ? bf16_to_f32(__builtin_amdgcn_raw_buffer_load_b16(rw, (int)voff, (int)so, 0))
                           : 0.f;
            }
          }
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const uint32_t so = (uint32_t)((erow(i, r) * d + j * 32) * 2);
            const float x = kMode == DW_ACCUMULATE ? old[r] + acc[i][j][r] : acc[i][j][r];
            if (decltype(kFull)::value || row_ok(i, r))
              __builtin_amdgcn_raw_buffer_store_b16(to_bf16(x), rw, (int)voff, (int)so, 0);
          }
        }
    };
    if (!partial && d0 + TILE <= d) store_tile(std::true_type{});
    else store_tile(std::false_type{});
  } else {
    // moments (and master) fp32 with row stride d, W bf16 with row stride ldw
    const __amdgpu_buffer_rsrc_t rm = make_rsrc(st.m + r0 * d, (uint64_t)rows * d * 4);
    const __amdgpu_buffer_rsrc_t rv = make_rsrc(st.v + r0 * d, (uint64_t)rows * d * 4);
    const __amdgpu_buffer_rsrc_t rp = make_rsrc(st.master ? st.master + r0 * d : st.m, st.master ? (uint64_t)rows * d * 4 : 0);
    const __amdgpu_buffer_rsrc_t rW = make_rsrc(st.W + r0 * st.ldw, (uint64_t)rows * st.ldw * 2);
    const bool has_master = st.master != nullptr;
    const uint32_t vo4 = (uint32_t)((lrow * d + dc) * 4);
    const uint32_t voW = (uint32_t)((lrow * st.ldw + dc) * 2);
    // as for the stores above: full tiles test nothing per element
    auto update_tile = [&](auto kFull) {
      constexpr bool kF = decltype(kFull)::value;
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
          if (!kF && !col_ok[j]) continue;
          // four consecutive rows at a time: all their loads first, then the updates and stores
#pragma unroll
          for (int rq = 0; rq < 4; ++rq) {
            float p[4], mo[4], vo[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int row = erow(i, rq * 4 + e);
              const uint32_t s4 = (uint32_t)((row * d + j * 32) * 4);
              const uint32_t sW = (uint32_t)((row * st.ldw + j * 32) * 2);
              mo[e] = vo[e] = p[e] = 0.f;
              if (kF || row_ok(i, rq * 4 + e)) {
                mo[e] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rm, (int)vo4, (int)s4, 0));
                vo[e] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rv, (int)vo4, (int)s4, 0));
                p[e] = has_master ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rp, (int)vo4, (int)s4, 0))
                                  : bf16_to_f32(__builtin_amdgcn_raw_buffer_load_b16(rW, (int)voW, (int)sW, 0));
              }
            }
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const int row = erow(i, rq * 4 + e);
              const uint32_t s4 = (uint32_t)((row * d + j * 32) * 4);
              const uint32_t sW = (uint32_t)((row * st.ldw + j * 32) * 2);
              if (!kF && !row_ok(i, rq * 4 + e)) continue;
              const float g = bf16_to_f32(to_bf16(acc[i][j][rq * 4 + e]));
              adamw_update(p[e], mo[e], vo[e], g, oc);
              __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, mo[e]), rm, (int)vo4, (int)s4, 0);
              __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, vo[e]), rv, (int)vo4, (int)s4, 0);
              if (has_master)
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, p[e]), rp, (int)vo4, (int)s4, 0);
              __builtin_amdgcn_raw_buffer_store_b16(to_bf16(p[e]), rW, (int)voW, (int)sW, 0);
            }
          }
        }
    };
    if (!partial && d0 + TILE <= d) update_tile(std::true_type{});
    else update_tile(std::false_type{});
  }
}

template <int kMode, int WM>
__global__ __launch_bounds__(Geo<WM>::NT, WM) void k_bwd_dw(const uint16_t* __restrict__ G, int vc, int ldt, int vs,
                                                           const uint16_t* __restrict__ Hv, int d,
                                                           const int* __restrict__ nv_ptr, int tm_count,
                                                           uint16_t* __restrict__ dW, int64_t v0,
                                                           AdamWState st, AdamWConst oc) {
  __shared__ __attribute__((aligned(16))) char smem[Geo<WM>::LDS];
  dw_tile<kMode, WM>(smem, (int)blockIdx.x, G, vc, ldt, vs, Hv, d, nv_ptr, tm_count, dW, v0, st, oc);
}

// K6: dH32[m][dd] (+)= sum_k G[m][k] Ws[k][dd] over the slab's k < vs; rows m < Nv. Ws = W + v0 ldw
// is the slab's first row, read K-major (transposing LDS reads); ws_rows = V - v0 rows follow.
// kz > 1 splits K in kz parts for launches with fewer output tiles than CUs: the blocks of part z
// (the z-th kz-th of the grid) accumulate into accumulator z, at dH32 + z (dH32b - dH32) (the
// parts follow each other), and the finalise adds the kz accumulators in a fixed order.
// One dH tile (block blk of a dH grid of `grid` blocks, smem the workgroup's LDS).
template <int WM>
__device__ __forceinline__ void dh_tile(char* smem, int blk, int grid, const uint16_t* __restrict__ G, int vc, int vs,
                                        const uint16_t* __restrict__ Ws, int64_t ldw, int64_t ws_rows, int d,
                                        const int* __restrict__ nv_ptr, float* __restrict__ dH32, int accumulate,
                                        int kz, float* __restrict__ dH32b, int acc_rows) {
  static_assert(Geo<WM>::TM == 384, "the tail slots and the finalise assume 384-row tiles");
  constexpr int TM = Geo<WM>::TM;
  const int nv = *nv_ptr;
  const int dt = (d + TILE - 1) / TILE, tm_live = (nv + TM - 1) / TM;
  // this block's tile, K part z of kzl, and the fp32 block it accumulates into (tile origin,
  // row stride, column of the tile's first column)
  int tm, tn, z, kzl;
  float* acc_tile;
  int ldacc, cb;
  if (kz > 1) {
    // the host split every tile's K into kz parts (launches with fewer tiles than CUs)
    const int g1 = grid / kz;
    z = blk / g1;
    kzl = kz;
    if (!band_tile(blk - z * g1, tm_live, dt, tm, tn)) return;
    acc_tile = (z ? dH32 + (int64_t)z * (dH32b - dH32) : dH32) + (int64_t)tm * TM * d;
    ldacc = d;
    cb = tn * TILE;
  } else {
    const int t = tm_live * dt, x = blk & 7, k = blk >> 3;
    const int c0 = dh_c0(x, t), n = dh_c0(x + 1, t) - c0, nmain = n & ~31, nt = n - nmain;
    const int kzt = dh_tail_fits(t, tm_live, d, acc_rows) ? dh_tail_parts(nt) : 1;
    int l, slot = 0;
    if (k < nmain) {
      l = c0 + k;
      z = 0;
      kzl = 1;
    } else {
      const int j = k - nmain;
      if (j >= kzt * nt) return;
      const int ti = j % nt;
      z = j / nt;
      kzl = kzt;
      l = c0 + nmain + ti;
      slot = dh_slot0(x, t) + (z - 1) * nt + ti;
    }
    dh_band_tile(l, tm_live, dt, tm, tn);
    if (z == 0) {
      acc_tile = dH32 + (int64_t)tm * TM * d;
      ldacc = d;
      cb = tn * TILE;
    } else {
      acc_tile = dH32 + (int64_t)tm_live * TM * d + (int64_t)slot * kDhSlot;
      ldacc = TILE;
      cb = 0;
    }
  }
  const int m0 = tm * TM, d0 = tn * TILE;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, wr = wave >> 2, wc = wave & 3;
  // K = the slab's vs ids; the last slice of a slab whose width is not a multiple of 64 is masked
  // (lanes past K load zeros), so no W row past the vocabulary is addressed. Half z covers
  // [k0, k0 + kzn), the first half a whole number of 64-wide slices.
  const int kt = (vs + KSLICE - 1) / KSLICE * KSLICE;
  const int kh = ((kt + kzl - 1) / kzl + KSLICE - 1) / KSLICE * KSLICE;
  const int k0 = z * kh;
  const int kzn = vs - k0 < kh ? vs - k0 : kh;
  f32x16_t acc[4][2];
  if (kzn > 0) {
    const Operand opa = dense_operand(G + (int64_t)m0 * vc + k0, nv - m0, vc);
    const Operand opb = kmajor_operand<TILE>(Ws + (int64_t)k0 * ldw + d0, ldw, ((uint64_t)(ws_rows - k0) * ldw - d0) * 2,
                                             d - d0);
    if (kzn % KSLICE == 0)
      mma_mainloop<121, OP_DENSE, OP_KMAJOR, WM, false>(acc, opa, opb, kzn, smem);
    else
      mma_mainloop<121, OP_DENSE, OP_KMAJOR, WM, true>(acc, opa, opb, kzn, smem);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = (f32x16_t){};
  }
  // Read-modify-write of the fp32 accumulator block through a buffer resource over this tile's
  // valid rows (rows past Nv read 0 and drop their stores): one 32-bit per-lane offset and a
  // wave-uniform row offset per element, so that only the accumulators occupy registers; one
  // 32-row block (32 values per lane) at a time, its loads in flight together.
  const int rows = nv - m0 < TM ? nv - m0 : TM;
  const __amdgpu_buffer_rsrc_t rd = make_rsrc(acc_tile, (uint64_t)rows * ldacc * 4);
  const int dc = d0 + wc * 64 + (lane & 31);      // column of dH (validity)
  const uint32_t voff = (uint32_t)(((wr * 128 + (lane >> 5) * 4) * ldacc + cb + wc * 64 + (lane & 31)) * 4);
  const bool col_ok[2] = {dc < d, dc + 32 < d};
  // (a column past D would be the next row's: never touched; tiles of whole 256-column blocks
  // test nothing per element, and the first slab's tiles read nothing)
  auto rmw = [&](auto kFull, auto kAcc) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      float old[2][16];
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const uint32_t so = (uint32_t)(((i * 32 + (r >> 2) * 8 + (r & 3)) * ldacc + j * 32) * 4);
          old[j][r] = (decltype(kAcc)::value && (decltype(kFull)::value || col_ok[j]))
                          ? __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rd, (int)voff, (int)so, 0))
                          : 0.f;
        }
#pragma unroll
      for (int j = 0; j < 2; ++j) {
        if (!decltype(kFull)::value && !col_ok[j]) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const uint32_t so = (uint32_t)(((i * 32 + (r >> 2) * 8 + (r & 3)) * ldacc + j * 32) * 4);
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, old[j][r] + acc[i][j][r]), rd,
                                                (int)voff, (int)so, 0);
        }
      }
    }
  };
  const bool full = d0 + TILE <= d;
  if (accumulate) {
    if (full) rmw(std::true_type{}, std::true_type{});
    else rmw(std::false_type{}, std::true_type{});
  } else {
    if (full) rmw(std::true_type{}, std::false_type{});
    else rmw(std::false_type{}, std::false_type{});
  }
}

template <int WM>
__global__ __launch_bounds__(Geo<WM>::NT, WM) void k_bwd_dh(const uint16_t* __restrict__ G, int vc, int vs,
                                                        const uint16_t* __restrict__ Ws, int64_t ldw,
                                                        int64_t ws_rows, int d,
                                                        const int* __restrict__ nv_ptr,
                                                        float* __restrict__ dH32, int accumulate, int kz,
                                                        float* __restrict__ dH32b, int acc_rows) {
  __shared__ __attribute__((aligned(16))) char smem[Geo<WM>::LDS];
  dh_tile<WM>(smem, (int)blockIdx.x, (int)gridDim.x, G, vc, vs, Ws, ldw, ws_rows, d, nv_ptr, dH32, accumulate, kz,
              dH32b, acc_rows);
}

// K7: dH[row] = bf16(dH32[pos[row]]) for valid rows, +0.0 for the others. 8 elements per thread.
__global__ __launch_bounds__(256) void k_dh_finalize(const float* __restrict__ dH32, int64_t part, int kz,
                                                     const int* __restrict__ pos, int64_t n, int d,
                                                     uint16_t* __restrict__ dH, float* __restrict__ dHf,
                                                     int has_slabs, const int* __restrict__ nv_ptr, int acc_rows) {
  // kz accumulators (the K parts of split dH launches), `part` elements apart, added in order;
  // with kz = 1, the slots of the tail tiles' K parts z = 1, 2, ... after part 0 (dh_tile)
  const int64_t e = ((int64_t)blockIdx.x * 256 + threadIdx.x) * 8;
  if (e >= n * d) return;
  const int64_t row = e / d;
  const int col = (int)(e - row * d);
  const int p = pos[row];
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
  auto add = [&](const float* q) {
    const float4 a2 = *reinterpret_cast<const float4*>(q);
    const float4 b2 = *reinterpret_cast<const float4*>(q + 4);
    a = make_float4(a.x + a2.x, a.y + a2.y, a.z + a2.z, a.w + a2.w);
    b = make_float4(b.x + b2.x, b.y + b2.y, b.z + b2.z, b.w + b2.w);
  };
  if (p >= 0 && has_slabs) {
    a = *reinterpret_cast<const float4*>(dH32 + (int64_t)p * d + col);
    b = *reinterpret_cast<const float4*>(dH32 + (int64_t)p * d + col + 4);
    for (int z = 1; z < kz; ++z) add(dH32 + z * part + (int64_t)p * d + col);
    if (kz == 1) {
      const int nv = *nv_ptr;
      const int tm_live = (nv + 383) / 384, dt = (d + TILE - 1) / TILE, t = tm_live * dt;
      if (dh_tail_fits(t, tm_live, d, acc_rows)) {
        const int tm = p / 384, tn = col / TILE;
        const int l = dh_band_index(tm, tn, tm_live, dt);
        int x = 0;
        while (x < 7 && dh_c0(x + 1, t) <= l) ++x;
        const int c0 = dh_c0(x, t), nmain = (dh_c0(x + 1, t) - c0) & ~31, nt = dh_c0(x + 1, t) - c0 - nmain;
        if (l - c0 >= nmain) {
          const int kzt = dh_tail_parts(nt), s0 = dh_slot0(x, t) + (l - c0 - nmain);
          const float* q = dH32 + (int64_t)tm_live * 384 * d + (int64_t)(p - tm * 384) * TILE + (col - tn * TILE);
          for (int z = 1; z < kzt; ++z) add(q + (int64_t)(s0 + (z - 1) * nt) * kDhSlot);
        }
      }
    }
  }
  if (dHf) {   // fp32 rows (a vocabulary shard's term of dH, to be summed over shards)
    store16_padded(dHf + e, __builtin_bit_cast(i32x4_t, a));
    store16_padded(dHf + e + 4, __builtin_bit_cast(i32x4_t, b));
  } else {
    store16_padded(dH + e, __builtin_bit_cast(i32x4_t,
        make_uint4(pack_bf16x2(a.x, a.y), pack_bf16x2(a.z, a.w), pack_bf16x2(b.x, b.y), pack_bf16x2(b.z, b.w))));
  }
}

__global__ __launch_bounds__(256) void k_zero16(uint4* __restrict__ p, int64_t n16) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n16) p[i] = make_uint4(0, 0, 0, 0);
}

// Standalone AdamW step over W [V, D] with the bf16 gradient dW (dense [V, D]; null = zero
// gradient): eight consecutive elements of one row per thread and iteration, 16-byte accesses.
__global__ __launch_bounds__(256) void k_adamw(int64_t v, int d, const uint16_t* __restrict__ dW,
                                               AdamWState st, AdamWConst oc) {
  const int cpr = d >> 3;
  const int64_t total = v * cpr;
  for (int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x; q < total; q += (int64_t)gridDim.x * 256) {
    const int64_t row = q / cpr;
    const int col = (int)(q - row * cpr) * 8;
    const int64_t o = row * d + col;
    i32x4_t wv = {0, 0, 0, 0};
    if (!st.master) wv = *reinterpret_cast<const i32x4_t*>(st.W + row * st.ldw + col);
    i32x4_t gv = {0, 0, 0, 0};
    if (dW) gv = *reinterpret_cast<const i32x4_t*>(dW + o);
    float p[8], mo[8], vo[8];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const float4 a = *reinterpret_cast<const float4*>(st.m + o + 4 * h);
      const float4 b = *reinterpret_cast<const float4*>(st.v + o + 4 * h);
      mo[4 * h] = a.x; mo[4 * h + 1] = a.y; mo[4 * h + 2] = a.z; mo[4 * h + 3] = a.w;
      vo[4 * h] = b.x; vo[4 * h + 1] = b.y; vo[4 * h + 2] = b.z; vo[4 * h + 3] = b.w;
      if (st.master) {
        const float4 c = *reinterpret_cast<const float4*>(st.master + o + 4 * h);
        p[4 * h] = c.x; p[4 * h + 1] = c.y; p[4 * h + 2] = c.z; p[4 * h + 3] = c.w;
      }
    }
    uint32_t wout[4];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t w2 = (uint32_t)wv[e >> 1], g2 = (uint32_t)gv[e >> 1];
      if (!st.master) p[e] = bf16_to_f32((e & 1) ? (w2 >> 16) : (w2 & 0xFFFFu));
      const float g = bf16_to_f32((e & 1) ? (g2 >> 16) : (g2 & 0xFFFFu));
      adamw_update(p[e], mo[e], vo[e], g, oc);
    }
#pragma unroll
    for (int e = 0; e < 4; ++e)
      wout[e] = pack_bf16x2(p[2 * e], p[2 * e + 1]);
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      *reinterpret_cast<float4*>(st.m + o + 4 * h) = make_float4(mo[4 * h], mo[4 * h + 1], mo[4 * h + 2], mo[4 * h + 3]);
      *reinterpret_cast<float4*>(st.v + o + 4 * h) = make_float4(vo[4 * h], vo[4 * h + 1], vo[4 * h + 2], vo[4 * h + 3]);
      if (st.master)
        *reinterpret_cast<float4*>(st.master + o + 4 * h) = make_float4(p[4 * h], p[4 * h + 1], p[4 * h + 2], p[4 * h + 3]);
    }
    *reinterpret_cast<i32x4_t*>(st.W + row * st.ldw + col) = i32x4_t{(int)wout[0], (int)wout[1], (int)wout[2], (int)wout[3]};
  }
}

// KD per-token loss: l = lse_s - sum of the token's Q partials (fixed order), for valid rows; terms
// (compact order) feed the mean / sum, per_token (row order, 0 on rows outside M) is the "none"
// output.
__global__ __launch_bounds__(256) void k_kd_terms(const float* __restrict__ qpart, int nq, int64_t ldq,
                                                  const int* __restrict__ pos, int64_t n,
                                                  const float* __restrict__ lse_s, float* __restrict__ terms,
                                                  float* __restrict__ per_token) {
  const int64_t row = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (row >= n) return;
  const int i = pos[row];
  if (i < 0) {
    if (per_token) per_token[row] = 0.f;
    return;
  }
  float q = 0.f;
  for (int k = 0; k < nq; ++k) q += qpart[k * ldq + i];
  const float l = lse_s[row] - q;
  terms[i] = l;
  if (per_token) per_token[row] = l;
}

// ---------------------------------------------------------------------------------------------
// Host side: validation, plan, workspace carve-up, launches, optional timing.
// ---------------------------------------------------------------------------------------------
enum KernelId { K_COMPACT = 0, K_FWD_STATS, K_COMBINE, K_LOSS, K_GATHER_H, K_BWD_G,
                K_BWD_DW, K_BWD_DH, K_DH_FINAL, K_ADAMW, K_SHARD_COMBINE, K_KD_P, K_KD_Q, K_KD_TERMS, K_MISC,
                K_COUNT };
const char* const kKernelNames[K_COUNT] = {"compact", "fwd_stats", "combine", "loss", "gather_h",
                                           "bwd_g", "bwd_dw", "bwd_dh", "dh_finalize", "adamw", "shard_combine",
                                           "kd_teacher_p", "kd_q", "kd_terms", "misc"};

struct Timing {
  std::mutex mu;
  bool on = false;
  static constexpr int kPool = 8192;
  std::vector<hipEvent_t> ev;   // 2 per record
  std::vector<int> kind;
  int used = 0;
};
Timing g_timing;

struct Plan {
  int64_t n, d, v, ldh, ldw, npad;
  int nt_max, vt_count, nparts, vt_count3;   // vt_count3: 384-id tiles
  int64_t vc, nslab;
  int64_t gw;                                // 384-id tiles of the forward's vocabulary groups
  int64_t rows_g;                            // rows of G and dH32: Npad rounded up to a 384-row tile
  // workspace offsets; idx, pos, Nv and the gathered rows Hv form a prefix both passes share
  size_t o_idx, o_pos, o_nv, o_hv, o_pm, o_ps, o_terms, fwd_bytes;
  size_t o_g, o_dh32, o_dh32b, bwd_bytes;    // o_dh32b: accumulator of the second K part (or 0)
  int dh_kz;                                 // K parts of the dH launches (1 to 8)
  int part_rows;                             // partial rows of the forward statistics
};

// the 12-wave forward in one launch: its partial rows (8 bytes per 384-id tile and token) take at
// most 2 D bytes per token
inline bool fwd_one_launch(const Plan& pl) {
  return pl.vt_count3 <= pl.d / 4 && (int64_t)pl.vt_count3 * pl.nt_max <= INT32_MAX;
}

// the forward statistics run on 12-wave tiles over the gathered rows Hv (left in the workspace)
inline bool fwd_gathers(const Plan& pl) {
  return pl.d % KSLICE == 0 && (int64_t)pl.vt_count3 * pl.nt_max <= INT32_MAX;
}

inline int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }

// Width, in tiles of tile_rows W rows, of the vocabulary groups the forward and G launches take
// in turn (each group by all token tiles): `tiles` split into equal groups whose W rows fit
// kGroupBytes, so that a group stays in the 256 MB MALL while the token tiles pass.
constexpr int64_t kGroupBytes = (int64_t)160 << 20;
inline int group_tiles(int64_t tiles, int64_t tile_rows, int64_t d) {
  const int64_t bytes = tiles * tile_rows * d * 2;
  const int64_t groups = std::max<int64_t>(1, (bytes + kGroupBytes - 1) / kGroupBytes);
  return (int)std::max<int64_t>(1, (tiles + groups - 1) / groups);
}

// Grid and group width of a launch in the order of xcd_tile: `tiles` vocabulary tiles by nt token
// tiles, in groups at most `width` tiles wide (rounded down to a multiple of 8).
struct TileOrder {
  unsigned grid;
  int gw;
};
inline TileOrder tile_order(int64_t tiles, int64_t nt, int64_t width) {
  const int64_t a = tiles & ~(int64_t)7, rem = tiles - a;
  return TileOrder{(unsigned)(a * nt + (rem ? 8 * rem * ((nt + 7) / 8) : 0)),
                   (int)std::max<int64_t>(8, std::min(width, a) & ~(int64_t)7)};
}

// Workgroup rounds of the dW launches over the whole vocabulary with slabs of r 384-id row tiles:
// a slab's ceil(vs / 384) x ceil(D / 256) tiles are cut evenly over the 8 XCDs of 32 CUs each.
int64_t dw_rounds(int64_t v, int64_t d, int64_t r) {
  const int64_t dt = (d + 255) / 256, vt = (v + 383) / 384;
  int64_t total = 0;
  for (int64_t t0 = 0; t0 < vt; t0 += r) {
    const int64_t tiles = std::min(r, vt - t0) * dt;
    total += ((tiles + 7) / 8 + 31) / 32;
  }
  return total;
}

// The slab width, among multiples of 768 ids from max(8192, 4 D) up to what the MALL rule allows
// (the slab's W rows within kGroupBytes, at most 24576 ids), that gives the dW launches the fewest
// workgroup rounds; vc (the rule's own width) unless another needs strictly fewer, and of those
// the widest. A head whose column tiles do not divide 256 (3584 wide: 14) leaves most of a last
// round idle in every slab at the rule's width.
int64_t whole_round_slab(int64_t v, int64_t d, int64_t vc) {
  const int64_t lo = std::max<int64_t>(8192, 4 * d);
  const int64_t hi = std::min(round_up(v, 768), std::max<int64_t>(vc, std::min<int64_t>(24576, kGroupBytes / (2 * d))));
  const int64_t c0 = dw_rounds(v, d, vc / 384);
  int64_t best = vc / 384, cost = c0;
  for (int64_t r = (lo + 767) / 768 * 2; r * 384 <= hi; r += 2) {
    const int64_t c = dw_rounds(v, d, r);
    if (c < cost || (c == cost && c < c0)) {   // r grows: of equal counts the widest
      best = r;
      cost = c;
    }
  }
  return best * 384;
}

lce_status_t make_plan(const lce_problem_t* p, Plan* pl, bool wide_slabs = true) {
  if (!p) return LCE_ERR_NULL;
  if ((p->flags & ~(LCE_FLAG_ACCUMULATE_DW | LCE_FLAG_REUSE_FORWARD)) != 0) return LCE_ERR_ARG;
  if (p->n < 0 || p->d < 1 || p->v < 1) return LCE_ERR_SHAPE;
  if (p->d % 8 != 0) return LCE_ERR_UNSUPPORTED;
  if (p->reduction != LCE_REDUCE_MEAN && p->reduction != LCE_REDUCE_SUM && p->reduction != LCE_REDUCE_NONE)
    return LCE_ERR_UNSUPPORTED;
  if (p->target_bytes != 4 && p->target_bytes != 8) return LCE_ERR_UNSUPPORTED;
  const int64_t ldh = p->ld_h ? p->ld_h : p->d, ldw = p->ld_w ? p->ld_w : p->d;
  if (ldh < p->d || ldw < p->d) return LCE_ERR_SHAPE;
  if (ldh % 8 != 0 || ldw % 8 != 0) return LCE_ERR_ALIGN;
  // 32-bit limits: token / vocabulary indices, and byte offsets inside one buffer resource
  if (p->n >= (int64_t)1 << 30 || p->v >= (int64_t)1 << 30 || p->d >= (int64_t)1 << 20) return LCE_ERR_SHAPE;
  if ((uint64_t)p->n * ldh * 2 > 0x7FFFFFFFull) return LCE_ERR_SHAPE;
  // byte offsets within one 384-row tile of W (bf16) and of the fp32 optimizer state
  if ((uint64_t)384 * ldw * 2 > 0x7FFFFFFFull || (uint64_t)384 * p->d * 4 > 0x7FFFFFFFull) return LCE_ERR_SHAPE;
  pl->n = p->n; pl->d = p->d; pl->v = p->v; pl->ldh = ldh; pl->ldw = ldw;
  pl->npad = round_up(p->n > 0 ? p->n : 1, TILE);
  pl->nt_max = (int)(pl->npad / TILE);
  pl->vt_count = (int)((p->v + TILE - 1) / TILE);
  pl->nparts = pl->vt_count < MAX_PARTS ? pl->vt_count : MAX_PARTS;
  pl->vt_count3 = (int)((p->v + 383) / 384);
  // backward vocabulary slab: about 4 D columns (at least 8192) keeps G at O(N D) while halving
  // the dH accumulator passes of a 2 D slab. Narrower heads take up to 24576 ids while the slab's
  // W rows fit kGroupBytes (they stay in the MALL while G's token tiles pass), which cuts their
  // fp32 accumulator passes further (the distillation calls keep the narrow slab: their teacher
  // probabilities take 4 bytes per slab id and token). A multiple of 16 tiles of 384 ids, so that
  // the dW launch of a 4096-wide head is whole rounds of workgroups on 256 CUs; for other widths
  // whole_round_slab picks the width whose dW launches leave the fewest idle CUs.
  int64_t vc = 4 * p->d;
  if (wide_slabs) vc = std::max<int64_t>(vc, std::min<int64_t>(24576, kGroupBytes / (2 * p->d) / 6144 * 6144));
  if (vc < 8192) vc = 8192;
  vc = round_up(vc, 16 * 384);
  // a multiple of 768 in any case: both 256- and 384-wide G tiles end inside a G row
  const int64_t vround = round_up(p->v, 768);
  if (vc > vround) vc = vround;
  // the forward's groups keep the rule's width (they only order its tiles; a wider group's W rows
  // leave the MALL)
  pl->gw = vc / 384;
  if (wide_slabs && vc < vround) vc = whole_round_slab(p->v, p->d, vc);
  pl->vc = vc;
  pl->nslab = (p->v + vc - 1) / vc;
  if ((uint64_t)TILE * pl->npad * 2 > 0x7FFFFFFFull || (uint64_t)TILE * vc * 2 > 0x7FFFFFFFull) return LCE_ERR_SHAPE;

  auto take = [](size_t& cur, size_t bytes) { size_t o = cur; cur += (bytes + 255) / 256 * 256; return o; };
  size_t cur = 0;
  pl->o_idx = take(cur, 4 * (size_t)pl->npad);
  pl->o_pos = take(cur, 4 * (size_t)pl->npad);
  pl->o_nv = take(cur, 256);
  // valid rows of H, gathered by the forward (12-wave statistics) and by the backward; a backward
  // with LCE_FLAG_REUSE_FORWARD finds the forward's here
  pl->o_hv = take(cur, 2 * (size_t)p->d * pl->npad);
  const size_t common = cur;
  // partial rows: 2 per partition (8-wave forward); one per 384-id tile while that is at most
  // 2 D bytes per token, else two sets of vc / 384 rows and a running pair (12-wave forward)
  const int64_t rows3 = fwd_one_launch(*pl) ? pl->vt_count3 : 2 * (vc / 384) + 1;
  const int64_t part_rows = 2 * pl->nparts > rows3 ? 2 * pl->nparts : rows3;
  pl->part_rows = (int)part_rows;
  pl->o_pm = take(cur, 4 * (size_t)part_rows * pl->npad);
  pl->o_ps = take(cur, 4 * (size_t)part_rows * pl->npad);
  pl->o_terms = take(cur, 4 * (size_t)pl->npad);
  pl->fwd_bytes = cur;
  cur = common;
  // G and the fp32 dH accumulators hold every row a 384-row dH tile can address (the tiles of
  // the last token rows reach past Npad), so that no access leaves its region
  pl->rows_g = round_up(pl->npad, 384);
  pl->o_g = take(cur, 2 * (size_t)pl->rows_g * vc);
  // dH launches with fewer 384 x 256 output tiles than the 256 CUs split K into kz parts (enough
  // to give every CU a block, at most 8), each accumulated in an accumulator of its own
  const int64_t dh_tiles = (pl->npad + 383) / 384 * ((p->d + TILE - 1) / TILE);
  pl->dh_kz = (int)std::min<int64_t>(8, (256 + dh_tiles - 1) / dh_tiles);
  const size_t part = 4 * (size_t)pl->rows_g * p->d;     // a multiple of 256 bytes
  pl->o_dh32 = take(cur, part * pl->dh_kz);
  pl->o_dh32b = pl->dh_kz > 1 ? pl->o_dh32 + part : 0;
  pl->bwd_bytes = cur;
  return LCE_OK;
}

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

lce_status_t make_adamw(const lce_adamw_t* o, AdamWConst* c) {
  if (!o) return LCE_ERR_NULL;
  if (o->reserved != 0 || o->step < 1) return LCE_ERR_ARG;
  if (!(o->lr >= 0.f && o->lr < INFINITY) || !(o->beta1 >= 0.f && o->beta1 < 1.f) ||
      !(o->beta2 >= 0.f && o->beta2 < 1.f) || !(o->eps >= 0.f && o->eps < INFINITY) ||
      !(o->weight_decay >= 0.f && o->weight_decay < INFINITY))
    return LCE_ERR_ARG;
  const double lr = o->lr, b1 = o->beta1, b2 = o->beta2;
  c->keep = (float)(1.0 - lr * (double)o->weight_decay);
  c->beta1 = o->beta1;
  c->omb1 = (float)(1.0 - b1);
  c->beta2 = o->beta2;
  c->omb2 = (float)(1.0 - b2);
  c->step_size = (float)(lr / (1.0 - pow(b1, (double)o->step)));
  c->inv_sqrt_bc2 = (float)(1.0 / sqrt(1.0 - pow(b2, (double)o->step)));
  c->eps = o->eps;
  return LCE_OK;
}

unsigned adamw_grid(int64_t v, int64_t d) {
  const int64_t chunks = v * (d / 8);
  const int64_t blocks = (chunks + 255) / 256;
  return (unsigned)(blocks < 16384 ? blocks : 16384);
}

struct Launcher {
  hipStream_t s;
  lce_status_t st = LCE_OK;
  // the kernel's arguments, converted to its parameter types, passed by address
  template <typename... KArgs>
  hipError_t launch(void (*kern)(KArgs...), dim3 grid, dim3 block, KArgs... a) {
    void* ptrs[sizeof...(KArgs) + 1] = {static_cast<void*>(&a)..., nullptr};
    return hipLaunchKernel(reinterpret_cast<const void*>(kern), grid, block, ptrs, 0, s);
  }
  template <typename... KArgs, typename... Args>
  void operator()(int kind, void (*kern)(KArgs...), dim3 grid, dim3 block, Args... args) {
    if (st != LCE_OK) return;
    if (grid.x == 0 || grid.y == 0 || grid.z == 0) return;
    int slot = -1;
    if (g_timing.on) {
      std::lock_guard<std::mutex> lk(g_timing.mu);
      if (g_timing.on && g_timing.used < Timing::kPool) {
        slot = g_timing.used++;
        g_timing.kind[slot] = kind;
      }
    }
    if (slot >= 0 && hipEventRecord(g_timing.ev[2 * slot], s) != hipSuccess) { st = LCE_ERR_HIP; return; }
    // the launch's own status, without reading (and clearing) the thread's last-error slot, which
    // may hold an earlier, unrelated call's error
    if (launch(kern, grid, block, static_cast<KArgs>(args)...) != hipSuccess) {
      st = LCE_ERR_HIP;
      return;
    }
    if (slot >= 0 && hipEventRecord(g_timing.ev[2 * slot + 1], s) != hipSuccess) st = LCE_ERR_HIP;
  }
};

// Which part of the vocabulary W holds: ids [v_begin, v_begin + p->v) of v_total (the whole
// vocabulary: v_begin = 0, v_total = p->v).
struct ShardInfo {
  int64_t v_total, v_begin;
};

lce_status_t shard_info(const lce_problem_t* p, const lce_shard_t* sh, ShardInfo* si) {
  if (!p || !sh) return LCE_ERR_NULL;
  if (sh->v_total < 1 || sh->v_total >= (int64_t)1 << 30 || sh->v_begin < 0 || p->v < 1 ||
      sh->v_begin + p->v > sh->v_total)
    return LCE_ERR_SHAPE;
  si->v_total = sh->v_total;
  si->v_begin = sh->v_begin;
  return LCE_OK;
}

// Partial rows that k_combine folds for one head: `count` rows of Npad from (m, s), after an
// optional running pair (run_m, run_s).
struct PartRows {
  const float* m;
  const float* s;
  int count;
  const float* run_m;
  const float* run_s;
};

// Vocabulary statistics of one head, in log2 units of the logits times scale2 / log2(e). With
// D % 64 == 0 and a gather buffer hv (Npad x D bf16), the valid rows of H are gathered and the
// 12-wave tiles run, in one launch or one per group of tiles as `layout` (the plan that sized the
// partial rows pm / ps) decides; otherwise the 8-wave partitions gather rows in their loop.
PartRows launch_fwd_stats(Launcher& L, const Plan& layout, const uint16_t* W, int64_t ldw, const uint16_t* H,
                          int64_t ldh, int d, const int* idx, const int* nv, uint16_t* hv, float* pm, float* ps,
                          float scale2) {
  const int v = (int)layout.v, npad = (int)layout.npad, nt_max = layout.nt_max;
  // (the same condition as fwd_gathers(layout) when d is the plan's own width)
  if (!(hv && d % KSLICE == 0 && (int64_t)layout.vt_count3 * nt_max <= INT32_MAX)) {
    L(K_FWD_STATS, k_fwd_stats<2>, dim3(nt_max * layout.nparts), dim3(NTHREADS), W, ldw, v, H, ldh, layout.n, idx,
      nv, d, layout.nparts, nt_max, layout.vt_count, pm, ps, npad, scale2);
    return PartRows{pm, ps, 2 * layout.nparts, nullptr, nullptr};
  }
  L(K_GATHER_H, k_gather_rows, dim3((unsigned)std::min<int64_t>(((int64_t)npad * (d / 8) + 255) / 256, 16384)),
    dim3(256), H, ldh, idx, nv, d, hv);
  const int gw = (int)(layout.vc / Geo<3>::TM);
  const int ntl = layout.vt_count3;
  if (fwd_one_launch(layout)) {
    // one launch: the groups only order the tiles (as wide as the slab rule's width, or narrower
    // where its W rows would not stay in the MALL)
    const TileOrder to = tile_order(ntl, nt_max, group_tiles(layout.gw, Geo<3>::TM, d));
    L(K_FWD_STATS, k_fwd_tile, dim3(to.grid), dim3(Geo<3>::NT), W, ldw, v, (const uint16_t*)hv,
      (int64_t)d, nv, d, 0, ntl, to.gw, nt_max, pm, ps, (const float*)nullptr, (const float*)nullptr, 0,
      (float*)nullptr, (float*)nullptr, 0, npad, scale2);
    return PartRows{pm, ps, ntl, nullptr, nullptr};
  }
  // one group per launch; row sets: parity 0 at rows [0, gw), parity 1 at [gw, 2 gw), the
  // running pair at row 2 gw
  const int ng = (ntl + gw - 1) / gw;
  const int64_t rs = (int64_t)gw * npad;
  float* run_m = pm + 2 * rs;
  float* run_s = ps + 2 * rs;
  for (int g = 0; g < ng; ++g) {
    const int tm0 = g * gw, wl = std::min(gw, ntl - tm0);
    const int64_t cur = (g & 1) * rs, prev = ((g + 1) & 1) * rs;
    const TileOrder to = tile_order(wl, nt_max, wl);
    L(K_FWD_STATS, k_fwd_tile, dim3(to.grid), dim3(Geo<3>::NT), W, ldw, v, (const uint16_t*)hv,
      (int64_t)d, nv, d, tm0, wl, to.gw, nt_max, pm + cur, ps + cur,
      g > 0 ? (const float*)(pm + prev) : (const float*)nullptr, (const float*)(ps + prev), gw, run_m, run_s,
      g == 1 ? 1 : 0, npad, scale2);
  }
  const int64_t last = ((ng - 1) & 1) * rs;
  return PartRows{pm + last, ps + last, ntl - (ng - 1) * gw, ng > 1 ? run_m : nullptr, run_s};
}

// The forward pass behind lce_forward and (tgt_part != null) lce_forward_shard.
lce_status_t forward_impl(const lce_problem_t* p, const ShardInfo* shard, const void* H, const void* W,
                          const void* targets, float* loss, float* lse, float* tgt_part, int32_t* n_valid,
                          int32_t* dev_status, void* workspace, size_t workspace_bytes, void* stream) {
  Plan pl;
  lce_status_t st = make_plan(p, &pl);
  if (st != LCE_OK) return st;
  const ShardInfo si = shard ? *shard : ShardInfo{pl.v, 0};
  if ((!shard && !loss) || (shard && !tgt_part) || !n_valid) return LCE_ERR_NULL;
  if (pl.n > 0 && (!H || !W || !targets || !lse || !workspace)) return LCE_ERR_NULL;
  if (pl.n > 0 && (!aligned16(H) || !aligned16(W) || ((uintptr_t)workspace & 255) != 0)) return LCE_ERR_ALIGN;
  if (pl.n > 0 && workspace_bytes < pl.fwd_bytes) return LCE_ERR_WORKSPACE;
  Launcher L{(hipStream_t)stream};
  const bool none = !shard && p->reduction == LCE_REDUCE_NONE;
  if (pl.n == 0) {
    L(K_MISC, k_fwd_empty, dim3(1), dim3(64), (none || shard) ? (float*)nullptr : loss, n_valid, dev_status);
    return L.st;
  }
  char* ws = (char*)workspace;
  int* idx = (int*)(ws + pl.o_idx);
  int* pos = (int*)(ws + pl.o_pos);
  int* nv = (int*)(ws + pl.o_nv);
  float* pm = (float*)(ws + pl.o_pm);
  float* ps = (float*)(ws + pl.o_ps);
  float* terms = (float*)(ws + pl.o_terms);
  const uint16_t* h = (const uint16_t*)H;
  const uint16_t* w = (const uint16_t*)W;

  // rows that are not valid get lse 0 and a zero per-token loss (or shard target logit)
  L(K_COMPACT, k_compact, dim3(1), dim3(1024), targets, p->target_bytes, pl.n, si.v_total, p->ignore_index,
    idx, pos, nv, n_valid, dev_status, lse, none ? loss : tgt_part);
  const PartRows pr = launch_fwd_stats(L, pl, w, pl.ldw, h, pl.ldh, (int)pl.d, (const int*)idx, (const int*)nv,
                                       (uint16_t*)(ws + pl.o_hv), pm, ps, kLog2e);
  L(K_COMBINE, k_combine, dim3((unsigned)((pl.n + kCombTok - 1) / kCombTok)), dim3(1024), h, pl.ldh, w, pl.ldw,
    targets, p->target_bytes, si.v_begin, pl.v, (const int*)idx, (const int*)nv, (int)pl.d, pr.count, pr.m, pr.s,
    (int)pl.npad, pr.run_m, pr.run_s, lse, terms, none ? loss : (float*)nullptr, tgt_part);
  if (!none && !shard) L(K_LOSS, k_loss, dim3(1), dim3(1024), (const float*)terms, (const int*)nv, p->reduction, loss);
  return L.st;
}

// Teacher head of the distillation loss, as the student's backward needs it: the teacher's
// probabilities are recomputed slab by slab into an fp32 buffer P [Vc][Npad] placed after the
// student's backward workspace.
struct KdArgs {
  const uint16_t* ht;
  int64_t ldht;
  const uint16_t* wt;
  int64_t ldwt;
  int dt;
  const float* lse_t;
  float scale2, inv_t;
  float* qpart;   // non-null: the student pass also writes the loss's Q partials (fused KD call)
};

inline size_t kd_p_bytes(const Plan& pl) { return (size_t)4 * pl.vc * pl.npad; }

// The teacher's valid rows gathered for its 12-wave probability pass (Npad x Dt bf16), when
// Dt % 64 == 0; placed after P.
inline size_t kd_hvt_bytes(const Plan& pl, int64_t dt) {
  return dt % KSLICE == 0 ? ((size_t)2 * dt * pl.npad + 255) / 256 * 256 : 0;
}

// Gather buffer for the 12-wave statistics of both distillation heads (Npad x max(Ds, Dt) bf16),
// placed in the teacher-probability buffer P (free before the slab loop), or null when P is
// too small (the 8-wave statistics then need none).
inline uint16_t* kd_stats_gather(const Plan& s, const Plan& t, char* p_buf) {
  const int64_t dmax = s.d > t.d ? s.d : t.d;
  return (size_t)2 * dmax * s.npad <= kd_p_bytes(s) ? (uint16_t*)p_buf : nullptr;
}

// The backward pass behind lce_backward (dW != null), lce_backward_adamw (adamw != null),
// lce_backward_shard (shard != null, fp32 dH term in dHf) and lce_kd_backward (kd != null).
lce_status_t backward_impl(const lce_problem_t* p, const ShardInfo* shard, const void* H, const void* W,
                           const void* targets, const float* lse, const int32_t* n_valid, const float* grad_loss,
                           void* dH, float* dHf, uint16_t* dW, const AdamWState* adamw, const AdamWConst* oc,
                           void* workspace, size_t workspace_bytes, void* stream, const KdArgs* kd = nullptr) {
  Plan pl;
  // the distillation calls keep the narrow slab of their own plan (make_kd_plan)
  lce_status_t st = make_plan(p, &pl, kd == nullptr);
  if (st != LCE_OK) return st;
  const ShardInfo si = shard ? *shard : ShardInfo{pl.v, 0};
  void* dH_any = dHf ? (void*)dHf : dH;
  if (!W || !grad_loss || (!n_valid && p->reduction == LCE_REDUCE_MEAN)) return LCE_ERR_NULL;
  if (pl.n > 0 && (!H || !targets || !lse || !dH_any || !workspace)) return LCE_ERR_NULL;
  if (!aligned16(W)) return LCE_ERR_ALIGN;
  if (pl.n > 0 && (!aligned16(H) || !aligned16(dH_any) || ((uintptr_t)workspace & 255) != 0)) return LCE_ERR_ALIGN;
  const size_t need = pl.bwd_bytes + (kd ? kd_p_bytes(pl) + kd_hvt_bytes(pl, kd->dt) : 0);
  if (pl.n > 0 && workspace_bytes < need) return LCE_ERR_WORKSPACE;
  const bool accumulate = (p->flags & LCE_FLAG_ACCUMULATE_DW) != 0;
  const AdamWState as = adamw ? *adamw : AdamWState{nullptr, 0, nullptr, nullptr, nullptr};
  const AdamWConst c = oc ? *oc : AdamWConst{};
  Launcher L{(hipStream_t)stream};
  if (pl.n == 0) {
    // no tokens: dW is zero, so the fused step is a step with a zero gradient
    if (adamw) {
      L(K_ADAMW, k_adamw, dim3(adamw_grid(pl.v, pl.d)), dim3(256), pl.v, (int)pl.d, (const uint16_t*)nullptr, as, c);
    } else if (!accumulate) {
      const int64_t n16 = pl.v * pl.d / 8;
      L(K_MISC, k_zero16, dim3((unsigned)((n16 + 255) / 256)), dim3(256), (uint4*)dW, n16);
    }
    return L.st;
  }
  char* ws = (char*)workspace;
  int* idx = (int*)(ws + pl.o_idx);
  int* pos = (int*)(ws + pl.o_pos);
  int* nv = (int*)(ws + pl.o_nv);
  uint16_t* hv = (uint16_t*)(ws + pl.o_hv);
  uint16_t* g = (uint16_t*)(ws + pl.o_g);
  float* dh32 = (float*)(ws + pl.o_dh32);
  float* dh32b = pl.dh_kz > 1 ? (float*)(ws + pl.o_dh32b) : nullptr;   // accumulator of K part 1 (parts follow)
  const uint16_t* h = (const uint16_t*)H;
  const uint16_t* w = (const uint16_t*)W;
  const int d = (int)pl.d, npad = (int)pl.npad, vc = (int)pl.vc;

  // with LCE_FLAG_REUSE_FORWARD the workspace holds the forward's valid-row list (and, when the
  // forward gathered them, the rows Hv); otherwise both are formed again
  const bool reuse = !kd && (p->flags & LCE_FLAG_REUSE_FORWARD) != 0;
  if (!reuse)
    L(K_COMPACT, k_compact, dim3(1), dim3(1024), targets, p->target_bytes, pl.n, si.v_total, p->ignore_index,
      idx, pos, nv, (int*)nullptr, (int*)nullptr, (float*)nullptr, (float*)nullptr);
  // Hv[i] = H[idx[i]] for i < Nv, zero rows up to round_up(Nv, 64)
  if (!(reuse && fwd_gathers(pl)))
    L(K_GATHER_H, k_gather_rows, dim3((unsigned)std::min<int64_t>((npad * (d / 8) + 255) / 256, 16384)), dim3(256),
      h, pl.ldh, (const int*)idx, (const int*)nv, d, hv);
  // KD: the teacher's valid rows for its 12-wave probability pass
  uint16_t* hvt = (kd && kd_hvt_bytes(pl, kd->dt) > 0) ? (uint16_t*)(ws + pl.bwd_bytes + kd_p_bytes(pl)) : nullptr;
  if (hvt)
    L(K_GATHER_H, k_gather_rows, dim3((unsigned)std::min<int64_t>(((int64_t)npad * (kd->dt / 8) + 255) / 256, 16384)),
      dim3(256), kd->ht, kd->ldht, (const int*)idx, (const int*)nv, kd->dt, hvt);
  const int dt = (d + TILE - 1) / TILE;
  const int dh_tiles = (int)((pl.npad + Geo<kDhWM>::TM - 1) / Geo<kDhWM>::TM);
  void (*dw_kernel)(const uint16_t*, int, int, int, const uint16_t*, int, const int*, int, uint16_t*, int64_t,
                    AdamWState, AdamWConst) =
      adamw ? k_bwd_dw<DW_ADAMW, kDwWM> : accumulate ? k_bwd_dw<DW_ACCUMULATE, kDwWM> : k_bwd_dw<DW_STORE, kDwWM>;
  for (int64_t s = 0; s < pl.nslab; ++s) {
    const int64_t v0 = s * pl.vc;
    const int vs = (int)(pl.v - v0 < pl.vc ? pl.v - v0 : pl.vc);
    const int tm = (vs + TILE - 1) / TILE;
    if (kd) {
      // teacher probabilities of this slab, then G = c (softmax(zs / T) - P) / T
      float* P = (float*)(ws + pl.bwd_bytes);
      if (hvt) {
        const int tmg = (vs + Geo<3>::TM - 1) / Geo<3>::TM;
        const TileOrder to = tile_order(tmg, pl.nt_max, group_tiles(tmg, Geo<3>::TM, kd->dt));
        L(K_KD_P, k_bwd_g<P_WRITE, 3>, dim3(to.grid), dim3(Geo<3>::NT), kd->wt, kd->ldwt, v0, vs,
          (const uint16_t*)hvt, (int64_t)kd->dt, pl.n, targets, p->target_bytes, (int64_t)0, (const int*)idx,
          (const int*)nv, kd->lse_t, grad_loss, (const int*)n_valid, p->reduction, kd->dt, tmg, (uint16_t*)nullptr, vc,
          npad, kd->scale2, kd->inv_t, P, (float*)nullptr, (int64_t)0, to.gw);
      } else {
        const TileOrder to = tile_order(tm, pl.nt_max, tm);
        L(K_KD_P, k_bwd_g<P_WRITE, 2>, dim3(to.grid), dim3(NTHREADS), kd->wt, kd->ldwt, v0, vs,
          kd->ht, kd->ldht, pl.n, targets, p->target_bytes, (int64_t)0, (const int*)idx, (const int*)nv, kd->lse_t,
          grad_loss, (const int*)n_valid, p->reduction, kd->dt, tm, (uint16_t*)nullptr, vc, npad,
          kd->scale2, kd->inv_t, P, (float*)nullptr, (int64_t)0, to.gw);
      }
      const TileOrder to = tile_order(tm, pl.nt_max, tm);
      if (kd->qpart)
        L(K_BWD_G, k_bwd_g<G_SOFT_Q, 2>, dim3(to.grid), dim3(NTHREADS), w, pl.ldw, v0, vs, h,
          pl.ldh, pl.n, targets, p->target_bytes, (int64_t)0, (const int*)idx, (const int*)nv, lse, grad_loss,
          (const int*)n_valid, p->reduction, d, tm, g, vc, npad, kd->scale2, kd->inv_t, P, kd->qpart,
          (int64_t)(2 * (v0 / TILE)), to.gw);
      else
        L(K_BWD_G, k_bwd_g<G_SOFT, 2>, dim3(to.grid), dim3(NTHREADS), w, pl.ldw, v0, vs, h,
          pl.ldh, pl.n, targets, p->target_bytes, (int64_t)0, (const int*)idx, (const int*)nv, lse, grad_loss,
          (const int*)n_valid, p->reduction, d, tm, g, vc, npad, kd->scale2, kd->inv_t, P, (float*)nullptr,
          (int64_t)0, to.gw);
    } else {
      if (d % KSLICE == 0) {
        const int tmg = (vs + Geo<kGWM>::TM - 1) / Geo<kGWM>::TM;
        const TileOrder to = tile_order(tmg, pl.nt_max, group_tiles(tmg, Geo<3>::TM, d));
        L(K_BWD_G, k_bwd_g<G_ONEHOT, kGWM>, dim3(to.grid), dim3(Geo<kGWM>::NT), w, pl.ldw, v0, vs,
          (const uint16_t*)hv, (int64_t)d, pl.n, targets, p->target_bytes, si.v_begin, (const int*)idx, (const int*)nv,
          lse, grad_loss, (const int*)n_valid, p->reduction, d, tmg, g, vc, npad, kLog2e, 1.f, (float*)nullptr,
          (float*)nullptr, (int64_t)0, to.gw);
      } else {
        const TileOrder to = tile_order(tm, pl.nt_max, tm);
        L(K_BWD_G, k_bwd_g<G_ONEHOT, 2>, dim3(to.grid), dim3(NTHREADS), w, pl.ldw, v0, vs, h,
          pl.ldh, pl.n, targets, p->target_bytes, si.v_begin, (const int*)idx, (const int*)nv, lse, grad_loss,
          (const int*)n_valid, p->reduction, d, tm, g, vc, npad, kLog2e, 1.f, (float*)nullptr, (float*)nullptr,
          (int64_t)0, to.gw);
      }
    }
    // split launches: kz copies of the banded grid; otherwise 8 XCDs x 32 CUs x (whole rounds of the
    // largest per-XCD share + one round for the split tail)
    const unsigned bdh = pl.dh_kz > 1 ? (unsigned)(pl.dh_kz * 8 * ((dh_tiles + 7) / 8) * dt)
                                      : (unsigned)(256 * (((int64_t)dh_tiles * dt + 7) / 8 / 32 + 1));
    const int tmw = (vs + Geo<kDwWM>::TM - 1) / Geo<kDwWM>::TM;
    const unsigned bdw = (unsigned)(8 * (((int64_t)tmw * dt + 7) / 8));
    // dH reads the slab's W rows before the dW launch, whose AdamW epilogue (in-backward step)
    // may update them; later slabs read only their own rows
    L(K_BWD_DH, k_bwd_dh<kDhWM>, dim3(bdh), dim3(Geo<kDhWM>::NT), (const uint16_t*)g, vc, vs, w + v0 * pl.ldw, pl.ldw,
      pl.v - v0, d, (const int*)nv, dh32, (int)(s > 0), pl.dh_kz, dh32b, (int)pl.rows_g);
    L(K_BWD_DW, dw_kernel, dim3(bdw), dim3(Geo<kDwWM>::NT), (const uint16_t*)g, vc, npad, vs, (const uint16_t*)hv, d,
      (const int*)nv, tmw, dW, v0, as, c);
  }
  const int64_t nthr = pl.n * pl.d / 8;
  L(K_DH_FINAL, k_dh_finalize, dim3((unsigned)((nthr + 255) / 256)), dim3(256), (const float*)dh32,
    (int64_t)pl.rows_g * d, pl.dh_kz, (const int*)pos, pl.n, d, (uint16_t*)dH, dHf, 1, (const int*)nv, (int)pl.rows_g);
  return L.st;
}

// ---- knowledge distillation --------------------------------------------------------------------
struct KdPlan {
  lce_problem_t ps, pt;   // student and teacher heads as LCE problems
  Plan s, t;
  float scale2, inv_t;
  size_t o_tgt, o_q, o_p, o_hvt, fwd_bytes, bwd_bytes;
  size_t f_q, f_tgt, fused_bytes;   // fused call: backward regions, P, then Q partials and scratch
};

lce_status_t make_kd_plan(const lce_kd_problem_t* p, KdPlan* k) {
  if (!p) return LCE_ERR_NULL;
  if (p->reserved != 0) return LCE_ERR_ARG;
  if (!(p->temperature > 0.f && p->temperature < INFINITY)) return LCE_ERR_ARG;
  if (p->flags & LCE_FLAG_REUSE_FORWARD) return LCE_ERR_ARG;   // the KD calls lay out their own workspace
  k->ps = lce_problem_t{p->n, p->ds, p->v, p->ld_hs, p->ld_ws, p->ignore_index, p->reduction, p->target_bytes, p->flags};
  k->pt = lce_problem_t{p->n, p->dt, p->v, p->ld_ht, p->ld_wt, p->ignore_index, p->reduction, p->target_bytes, 0};
  lce_status_t st = make_plan(&k->ps, &k->s, false);
  if (st != LCE_OK) return st;
  st = make_plan(&k->pt, &k->t, false);
  if (st != LCE_OK) return st;
  k->scale2 = (float)(1.4426950408889634 / (double)p->temperature);
  k->inv_t = (float)(1.0 / (double)p->temperature);
  // forward: the student plan's forward regions (index arrays, partials, terms; the teacher's
  // partials have the same shape), then target-logit scratch, Q partials and P
  auto up = [](size_t x) { return (x + 255) / 256 * 256; };
  size_t cur = up(k->s.fwd_bytes);
  k->o_tgt = cur;
  cur += up(4 * (size_t)k->s.npad);
  k->o_q = cur;
  cur += up((size_t)4 * 2 * k->s.vt_count * k->s.npad);
  k->o_p = cur;
  cur += up(kd_p_bytes(k->s));
  k->o_hvt = cur;
  cur += kd_hvt_bytes(k->s, k->t.d);
  k->fwd_bytes = cur;
  k->bwd_bytes = k->s.bwd_bytes + kd_p_bytes(k->s) + kd_hvt_bytes(k->s, k->t.d);
  cur = up(k->bwd_bytes);
  k->f_q = cur;
  cur += up((size_t)4 * 2 * k->s.vt_count * k->s.npad);
  k->f_tgt = cur;
  cur += up(4 * (size_t)k->s.npad);
  k->fused_bytes = cur;
  return LCE_OK;
}

// Forward and backward of the KD loss in one call (the upstream gradient is read on the device
// when the gradient kernels run): both heads' statistics, then per slab one teacher pass and one
// student pass that writes G and the loss's Q partials together.
lce_status_t kd_fused_impl(const lce_kd_problem_t* p, const void* Hs, const void* Ws, const void* Ht,
                           const void* Wt, const void* targets, const float* grad_loss, float* loss, float* lse_s,
                           float* lse_t, int32_t* n_valid, int32_t* dev_status, void* dHs, void* dWs,
                           void* workspace, size_t workspace_bytes, void* stream) {
  KdPlan k;
  lce_status_t st = make_kd_plan(p, &k);
  if (st != LCE_OK) return st;
  const Plan& pl = k.s;
  if (!loss || !n_valid || !grad_loss || !dWs) return LCE_ERR_NULL;
  if (!aligned16(dWs)) return LCE_ERR_ALIGN;
  if (pl.n > 0 && (!Hs || !Ws || !Ht || !Wt || !targets || !lse_s || !lse_t || !dHs || !workspace))
    return LCE_ERR_NULL;
  if (pl.n > 0 && (!aligned16(Hs) || !aligned16(Ws) || !aligned16(Ht) || !aligned16(Wt) || !aligned16(dHs) ||
                   ((uintptr_t)workspace & 255) != 0))
    return LCE_ERR_ALIGN;
  if (pl.n > 0 && workspace_bytes < k.fused_bytes) return LCE_ERR_WORKSPACE;
  const bool none = p->reduction == LCE_REDUCE_NONE;
  if (pl.n == 0) {
    Launcher L{(hipStream_t)stream};
    L(K_MISC, k_fwd_empty, dim3(1), dim3(64), none ? (float*)nullptr : loss, n_valid, dev_status);
    if (L.st != LCE_OK) return L.st;
    return backward_impl(&k.ps, nullptr, Hs, Ws, targets, lse_s, n_valid, grad_loss, dHs, nullptr,
                         (uint16_t*)dWs, nullptr, nullptr, workspace, workspace_bytes, stream);
  }
  char* ws = (char*)workspace;
  int* idx = (int*)(ws + pl.o_idx);
  int* pos = (int*)(ws + pl.o_pos);
  int* nv = (int*)(ws + pl.o_nv);
  float* pm = (float*)(ws + pl.o_pm);
  float* ps = (float*)(ws + pl.o_ps);
  float* tgt = (float*)(ws + k.f_tgt);
  float* qpart = (float*)(ws + k.f_q);
  const uint16_t* hs = (const uint16_t*)Hs;
  const uint16_t* wsm = (const uint16_t*)Ws;
  const uint16_t* ht = (const uint16_t*)Ht;
  const uint16_t* wt = (const uint16_t*)Wt;
  const Plan& tp = k.t;
  const int npad = (int)pl.npad;
  {
    Launcher L{(hipStream_t)stream};
    L(K_COMPACT, k_compact, dim3(1), dim3(1024), targets, p->target_bytes, pl.n, pl.v, p->ignore_index,
      idx, pos, nv, n_valid, dev_status, lse_s, lse_t);
    // the statistics' row gathers use the P buffer, free until the slab loop
    uint16_t* hvk = kd_stats_gather(pl, tp, ws + pl.bwd_bytes);
    const PartRows pt = launch_fwd_stats(L, pl, wt, tp.ldw, ht, tp.ldh, (int)tp.d, (const int*)idx, (const int*)nv, hvk,
                                         pm, ps, k.scale2);
    L(K_COMBINE, k_combine, dim3((unsigned)((pl.n + kCombTok - 1) / kCombTok)), dim3(1024), ht, tp.ldh, wt, tp.ldw, targets,
      p->target_bytes, (int64_t)0, (int64_t)0, (const int*)idx, (const int*)nv, (int)tp.d, pt.count, pt.m, pt.s, npad,
      pt.run_m, pt.run_s, lse_t, (float*)nullptr, (float*)nullptr, tgt);
    const PartRows pq = launch_fwd_stats(L, pl, wsm, pl.ldw, hs, pl.ldh, (int)pl.d, (const int*)idx, (const int*)nv, hvk,
                                         pm, ps, k.scale2);
    L(K_COMBINE, k_combine, dim3((unsigned)((pl.n + kCombTok - 1) / kCombTok)), dim3(1024), hs, pl.ldh, wsm, pl.ldw, targets,
      p->target_bytes, (int64_t)0, (int64_t)0, (const int*)idx, (const int*)nv, (int)pl.d, pq.count, pq.m, pq.s, npad,
      pq.run_m, pq.run_s, lse_s, (float*)nullptr, (float*)nullptr, tgt);
    if (L.st != LCE_OK) return L.st;
  }
  const KdArgs kd{ht, tp.ldh, wt, tp.ldw, (int)tp.d, lse_t, k.scale2, k.inv_t, qpart};
  st = backward_impl(&k.ps, nullptr, Hs, Ws, targets, lse_s, n_valid, grad_loss, dHs, nullptr, (uint16_t*)dWs,
                     nullptr, nullptr, workspace, workspace_bytes, stream, &kd);
  if (st != LCE_OK) return st;
  // the backward's workspace (idx, pos, Nv) is still valid; the per-token terms reuse the
  // student-statistics region, free again
  Launcher L{(hipStream_t)stream};
  float* terms = (float*)(ws + pl.o_terms);
  L(K_KD_TERMS, k_kd_terms, dim3((unsigned)((pl.n + 255) / 256)), dim3(256), (const float*)qpart,
    2 * pl.vt_count, (int64_t)npad, (const int*)pos, pl.n, (const float*)lse_s, terms, none ? loss : (float*)nullptr);
  if (!none) L(K_LOSS, k_loss, dim3(1), dim3(1024), (const float*)terms, (const int*)nv, p->reduction, loss);
  return L.st;
}

lce_status_t kd_forward_impl(const lce_kd_problem_t* p, const void* Hs, const void* Ws, const void* Ht,
                             const void* Wt, const void* targets, float* loss, float* lse_s, float* lse_t,
                             int32_t* n_valid, int32_t* dev_status, void* workspace, size_t workspace_bytes,
                             void* stream) {
  KdPlan k;
  lce_status_t st = make_kd_plan(p, &k);
  if (st != LCE_OK) return st;
  const Plan& pl = k.s;
  if (!loss || !n_valid) return LCE_ERR_NULL;
  if (pl.n > 0 && (!Hs || !Ws || !Ht || !Wt || !targets || !lse_s || !lse_t || !workspace)) return LCE_ERR_NULL;
  if (pl.n > 0 && (!aligned16(Hs) || !aligned16(Ws) || !aligned16(Ht) || !aligned16(Wt) ||
                   ((uintptr_t)workspace & 255) != 0))
    return LCE_ERR_ALIGN;
  if (pl.n > 0 && workspace_bytes < k.fwd_bytes) return LCE_ERR_WORKSPACE;
  Launcher L{(hipStream_t)stream};
  const bool none = p->reduction == LCE_REDUCE_NONE;
  if (pl.n == 0) {
    L(K_MISC, k_fwd_empty, dim3(1), dim3(64), none ? (float*)nullptr : loss, n_valid, dev_status);
    return L.st;
  }
  char* ws = (char*)workspace;
  int* idx = (int*)(ws + pl.o_idx);
  int* pos = (int*)(ws + pl.o_pos);
  int* nv = (int*)(ws + pl.o_nv);
  float* pm = (float*)(ws + pl.o_pm);
  float* ps = (float*)(ws + pl.o_ps);
  float* terms = (float*)(ws + pl.o_terms);
  float* tgt = (float*)(ws + k.o_tgt);
  float* qpart = (float*)(ws + k.o_q);
  float* P = (float*)(ws + k.o_p);
  const uint16_t* hs = (const uint16_t*)Hs;
  const uint16_t* wsm = (const uint16_t*)Ws;
  const uint16_t* ht = (const uint16_t*)Ht;
  const uint16_t* wt = (const uint16_t*)Wt;
  const int npad = (int)pl.npad, vc = (int)pl.vc;

  L(K_COMPACT, k_compact, dim3(1), dim3(1024), targets, p->target_bytes, pl.n, pl.v, p->ignore_index,
    idx, pos, nv, n_valid, dev_status, lse_s, lse_t);
  // log-sum-exp of both heads' logits / T (no target logit: an empty id range)
  const Plan& tp = k.t;
  // the statistics' row gathers use the P buffer, free until the slab loop
  uint16_t* hvk = kd_stats_gather(pl, tp, (char*)P);
  const PartRows pt = launch_fwd_stats(L, pl, wt, tp.ldw, ht, tp.ldh, (int)tp.d, (const int*)idx, (const int*)nv, hvk,
                                       pm, ps, k.scale2);
  L(K_COMBINE, k_combine, dim3((unsigned)((pl.n + kCombTok - 1) / kCombTok)), dim3(1024), ht, tp.ldh, wt, tp.ldw, targets,
    p->target_bytes, (int64_t)0, (int64_t)0, (const int*)idx, (const int*)nv, (int)tp.d, pt.count, pt.m, pt.s, npad,
    pt.run_m, pt.run_s, lse_t, terms, (float*)nullptr, tgt);
  const PartRows pq = launch_fwd_stats(L, pl, wsm, pl.ldw, hs, pl.ldh, (int)pl.d, (const int*)idx, (const int*)nv, hvk,
                                       pm, ps, k.scale2);
  L(K_COMBINE, k_combine, dim3((unsigned)((pl.n + kCombTok - 1) / kCombTok)), dim3(1024), hs, pl.ldh, wsm, pl.ldw, targets,
    p->target_bytes, (int64_t)0, (int64_t)0, (const int*)idx, (const int*)nv, (int)pl.d, pq.count, pq.m, pq.s, npad,
    pq.run_m, pq.run_s, lse_s, terms, (float*)nullptr, tgt);
  // per slab: teacher probabilities P, then the student's sum_v P zs / T per token and tile
  uint16_t* hvt = kd_hvt_bytes(pl, tp.d) > 0 ? (uint16_t*)(ws + k.o_hvt) : nullptr;
  if (hvt)
    L(K_GATHER_H, k_gather_rows, dim3((unsigned)std::min<int64_t>(((int64_t)npad * (tp.d / 8) + 255) / 256, 16384)),
      dim3(256), ht, tp.ldh, (const int*)idx, (const int*)nv, (int)tp.d, hvt);
  for (int64_t s = 0; s < pl.nslab; ++s) {
    const int64_t v0 = s * pl.vc;
    const int vs = (int)(pl.v - v0 < pl.vc ? pl.v - v0 : pl.vc);
    const int tm = (vs + TILE - 1) / TILE;
    if (hvt) {
      const int tmg = (vs + Geo<3>::TM - 1) / Geo<3>::TM;
      const TileOrder to = tile_order(tmg, pl.nt_max, group_tiles(tmg, Geo<3>::TM, tp.d));
      L(K_KD_P, k_bwd_g<P_WRITE, 3>, dim3(to.grid), dim3(Geo<3>::NT), wt, tp.ldw, v0, vs,
        (const uint16_t*)hvt, tp.d, pl.n, targets, p->target_bytes, (int64_t)0, (const int*)idx, (const int*)nv,
        (const float*)lse_t, (const float*)nullptr, (const int*)nullptr, p->reduction, (int)tp.d, tmg,
        (uint16_t*)nullptr, vc, npad, k.scale2, k.inv_t, P, (float*)nullptr, (int64_t)0, to.gw);
    } else {
      const TileOrder to = tile_order(tm, pl.nt_max, tm);
      L(K_KD_P, k_bwd_g<P_WRITE, 2>, dim3(to.grid), dim3(NTHREADS), wt, tp.ldw, v0, vs, ht, tp.ldh,
        pl.n, targets, p->target_bytes, (int64_t)0, (const int*)idx, (const int*)nv, (const float*)lse_t,
        (const float*)nullptr, (const int*)nullptr, p->reduction, (int)tp.d, tm, (uint16_t*)nullptr, vc,
        npad, k.scale2, k.inv_t, P, (float*)nullptr, (int64_t)0, to.gw);
    }
    const TileOrder to = tile_order(tm, pl.nt_max, tm);
    L(K_KD_Q, k_bwd_g<Q_SOFT, 2>, dim3(to.grid), dim3(NTHREADS), wsm, pl.ldw, v0, vs, hs, pl.ldh,
      pl.n, targets, p->target_bytes, (int64_t)0, (const int*)idx, (const int*)nv, (const float*)lse_s,
      (const float*)nullptr, (const int*)nullptr, p->reduction, (int)pl.d, tm, (uint16_t*)nullptr, vc,
      npad, k.scale2, k.inv_t, P, qpart, (int64_t)(2 * (v0 / TILE)), to.gw);
  }
  L(K_KD_TERMS, k_kd_terms, dim3((unsigned)((pl.n + 255) / 256)), dim3(256), (const float*)qpart,
    2 * pl.vt_count, (int64_t)npad, (const int*)pos, pl.n, (const float*)lse_s, terms, none ? loss : (float*)nullptr);
  if (!none) L(K_LOSS, k_loss, dim3(1), dim3(1024), (const float*)terms, (const int*)nv, p->reduction, loss);
  return L.st;
}

}  // namespace

extern "C" {

const char* lce_status_string(lce_status_t s) {
  switch (s) {
    case LCE_OK: return "ok";
    case LCE_ERR_NULL: return "required pointer is NULL";
    case LCE_ERR_SHAPE: return "invalid or too large shape / stride";
    case LCE_ERR_ALIGN: return "pointer, stride or workspace misaligned";
    case LCE_ERR_UNSUPPORTED: return "unsupported configuration (d % 8, reduction or target width)";
    case LCE_ERR_WORKSPACE: return "workspace too small";
    case LCE_ERR_HIP: return "HIP runtime or kernel launch failure";
    case LCE_ERR_ARG: return "invalid argument";
  }
  return "unknown status";
}

lce_status_t lce_plan_info(const lce_problem_t* p, lce_plan_info_t* out) {
  Plan pl;
  lce_status_t st = make_plan(p, &pl);
  if (st != LCE_OK) return st;
  if (!out) return LCE_ERR_NULL;
  out->npad = pl.npad;
  out->rows_g = pl.rows_g;
  out->vc = pl.vc;
  out->nslab = pl.nslab;
  out->dh_kz = pl.dh_kz;
  out->part_rows = pl.part_rows;
  out->fwd_gathers = fwd_gathers(pl) ? 1 : 0;
  out->fwd_one_launch = fwd_one_launch(pl) ? 1 : 0;
  out->o_idx = (int64_t)pl.o_idx;
  out->o_pos = (int64_t)pl.o_pos;
  out->o_nv = (int64_t)pl.o_nv;
  out->o_hv = (int64_t)pl.o_hv;
  out->o_pm = (int64_t)pl.o_pm;
  out->o_ps = (int64_t)pl.o_ps;
  out->o_terms = (int64_t)pl.o_terms;
  out->fwd_bytes = (int64_t)pl.fwd_bytes;
  out->o_g = (int64_t)pl.o_g;
  out->o_dh32 = (int64_t)pl.o_dh32;
  out->o_dh32b = (int64_t)pl.o_dh32b;
  out->bwd_bytes = (int64_t)pl.bwd_bytes;
  return LCE_OK;
}

// The device address of `scratch` on the current device, taken once per device (with that
// device current) and kept: every call on a GPU then shares that GPU's copy.
struct ScratchAddrs {
  std::mutex mu;
  static constexpr int kMaxDevices = 64;
  void* ptr[kMaxDevices] = {};
};
ScratchAddrs g_scratch;

lce_status_t noalloc_scratch(void* stream, void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= ScratchAddrs::kMaxDevices) return LCE_ERR_HIP;
  if (stream) {
    hipDevice_t sdev = -1;
    if (hipStreamGetDevice((hipStream_t)stream, &sdev) != hipSuccess) return LCE_ERR_HIP;
    if (sdev != dev) return LCE_ERR_ARG;   // the stream must belong to the current device
  }
  std::lock_guard<std::mutex> lk(g_scratch.mu);
  if (!g_scratch.ptr[dev]) {
    void* a = nullptr;
    if (hipGetSymbolAddress(&a, HIP_SYMBOL(scratch)) != hipSuccess || !a) return LCE_ERR_HIP;
    g_scratch.ptr[dev] = a;
  }
  *out = g_scratch.ptr[dev];
  return LCE_OK;
}

lce_status_t lce_workspace_size(const lce_problem_t* p, size_t* fwd_bytes, size_t* bwd_bytes) {
  Plan pl;
  lce_status_t st = make_plan(p, &pl);
  if (st != LCE_OK) return st;
  if (fwd_bytes) *fwd_bytes = pl.fwd_bytes;
  if (bwd_bytes) *bwd_bytes = pl.bwd_bytes;
  return LCE_OK;
}

lce_status_t lce_forward(const lce_problem_t* p, const void* H, const void* W, const void* targets,
                         float* loss, float* lse, int32_t* n_valid, int32_t* dev_status,
                         void* workspace, size_t workspace_bytes, void* stream) {
  return forward_impl(p, nullptr, H, W, targets, loss, lse, nullptr, n_valid, dev_status, workspace,
                      workspace_bytes, stream);
}

lce_status_t lce_forward_noalloc(const lce_problem_t* p, const void* H, const void* W, const void* targets,
                                 float* loss, float* lse, int32_t* n_valid, int32_t* dev_status, void* stream) {
  Plan pl;
  lce_status_t st = make_plan(p, &pl);
  if (st != LCE_OK) return st;
  if (pl.fwd_bytes > (size_t)LCE_NOALLOC_SCRATCH_BYTES) return LCE_ERR_WORKSPACE;
  void* ws = nullptr;
  st = noalloc_scratch(stream, &ws);
  if (st != LCE_OK) return st;
  // nothing of the previous call's contents is read: every region is written before it is used
  return forward_impl(p, nullptr, H, W, targets, loss, lse, nullptr, n_valid, dev_status, ws,
                      (size_t)LCE_NOALLOC_SCRATCH_BYTES, stream);
}

lce_status_t lce_forward_shard(const lce_problem_t* p, const lce_shard_t* shard, const void* H, const void* W,
                               const void* targets, float* lse_part, float* tgt_part, int32_t* n_valid,
                               int32_t* dev_status, void* workspace, size_t workspace_bytes, void* stream) {
  ShardInfo si;
  lce_status_t st = shard_info(p, shard, &si);
  if (st != LCE_OK) return st;
  return forward_impl(p, &si, H, W, targets, nullptr, lse_part, tgt_part, n_valid, dev_status, workspace,
                      workspace_bytes, stream);
}

lce_status_t lce_combine_shards(const lce_problem_t* p, int32_t n_shards, const float* lse_parts,
                                const float* tgt_parts, const void* targets, float* loss, float* lse,
                                int32_t* n_valid, int32_t* dev_status, void* workspace, size_t workspace_bytes,
                                void* stream) {
  Plan pl;
  lce_status_t st = make_plan(p, &pl);
  if (st != LCE_OK) return st;
  if (n_shards < 1 || n_shards > 4096) return LCE_ERR_ARG;
  if (!loss || !n_valid) return LCE_ERR_NULL;
  if (pl.n > 0 && (!lse_parts || !tgt_parts || !targets || !lse || !workspace)) return LCE_ERR_NULL;
  if (pl.n > 0 && ((uintptr_t)workspace & 255) != 0) return LCE_ERR_ALIGN;
  if (pl.n > 0 && workspace_bytes < pl.fwd_bytes) return LCE_ERR_WORKSPACE;
  Launcher L{(hipStream_t)stream};
  const bool none = p->reduction == LCE_REDUCE_NONE;
  if (pl.n == 0) {
    L(K_MISC, k_fwd_empty, dim3(1), dim3(64), none ? (float*)nullptr : loss, n_valid, dev_status);
    return L.st;
  }
  char* ws = (char*)workspace;
  int* idx = (int*)(ws + pl.o_idx);
  int* pos = (int*)(ws + pl.o_pos);
  int* nv = (int*)(ws + pl.o_nv);
  float* terms = (float*)(ws + pl.o_terms);
  L(K_COMPACT, k_compact, dim3(1), dim3(1024), targets, p->target_bytes, pl.n, pl.v, p->ignore_index,
    idx, pos, nv, n_valid, dev_status, lse, none ? loss : (float*)nullptr);
  L(K_SHARD_COMBINE, k_shard_combine, dim3((unsigned)((pl.n + 255) / 256)), dim3(256), (int)n_shards, lse_parts,
    tgt_parts, pl.n, (const int*)idx, (const int*)nv, lse, terms, none ? loss : (float*)nullptr);
  if (!none) L(K_LOSS, k_loss, dim3(1), dim3(1024), (const float*)terms, (const int*)nv, p->reduction, loss);
  return L.st;
}

lce_status_t lce_backward(const lce_problem_t* p, const void* H, const void* W, const void* targets,
                          const float* lse, const int32_t* n_valid, const float* grad_loss,
                          void* dH, void* dW, void* workspace, size_t workspace_bytes, void* stream) {
  if (!dW) return LCE_ERR_NULL;
  if (!aligned16(dW)) return LCE_ERR_ALIGN;
  return backward_impl(p, nullptr, H, W, targets, lse, n_valid, grad_loss, dH, nullptr, (uint16_t*)dW, nullptr,
                       nullptr, workspace, workspace_bytes, stream);
}

lce_status_t lce_backward_shard(const lce_problem_t* p, const lce_shard_t* shard, const void* H, const void* W,
                                const void* targets, const float* lse, const int32_t* n_valid,
                                const float* grad_loss, float* dH_part, void* dW, void* workspace,
                                size_t workspace_bytes, void* stream) {
  ShardInfo si;
  lce_status_t st = shard_info(p, shard, &si);
  if (st != LCE_OK) return st;
  if (!dW || (p->n > 0 && !dH_part)) return LCE_ERR_NULL;
  if (!aligned16(dW)) return LCE_ERR_ALIGN;
  return backward_impl(p, &si, H, W, targets, lse, n_valid, grad_loss, nullptr, dH_part, (uint16_t*)dW, nullptr,
                       nullptr, workspace, workspace_bytes, stream);
}

lce_status_t lce_adamw_step(int64_t v, int64_t d, int64_t ld_w, void* W, const void* dW, float* exp_avg,
                            float* exp_avg_sq, float* W_master, const lce_adamw_t* opt, void* stream) {
  AdamWConst c;
  lce_status_t st = make_adamw(opt, &c);
  if (st != LCE_OK) return st;
  const int64_t ldw = ld_w ? ld_w : d;
  if (v < 1 || d < 8 || ldw < d || v >= (int64_t)1 << 30 || d >= (int64_t)1 << 20) return LCE_ERR_SHAPE;
  if (d % 8 != 0) return LCE_ERR_UNSUPPORTED;
  if (ldw % 8 != 0) return LCE_ERR_ALIGN;
  if (!W || !exp_avg || !exp_avg_sq) return LCE_ERR_NULL;
  if (!aligned16(W) || !aligned16(exp_avg) || !aligned16(exp_avg_sq) || (dW && !aligned16(dW)) ||
      (W_master && !aligned16(W_master)))
    return LCE_ERR_ALIGN;
  AdamWState as{(uint16_t*)W, ldw, exp_avg, exp_avg_sq, W_master};
  Launcher L{(hipStream_t)stream};
  L(K_ADAMW, k_adamw, dim3(adamw_grid(v, d)), dim3(256), v, (int)d, (const uint16_t*)dW, as, c);
  return L.st;
}

lce_status_t lce_backward_adamw(const lce_problem_t* p, const void* H, void* W, const void* targets,
                                const float* lse, const int32_t* n_valid, const float* grad_loss, void* dH,
                                float* exp_avg, float* exp_avg_sq, float* W_master, const lce_adamw_t* opt,
                                void* workspace, size_t workspace_bytes, void* stream) {
  AdamWConst c;
  lce_status_t st = make_adamw(opt, &c);
  if (st != LCE_OK) return st;
  if (!p) return LCE_ERR_NULL;
  if (p->flags & LCE_FLAG_ACCUMULATE_DW) return LCE_ERR_ARG;
  if (!exp_avg || !exp_avg_sq) return LCE_ERR_NULL;
  if (!aligned16(exp_avg) || !aligned16(exp_avg_sq) || (W_master && !aligned16(W_master))) return LCE_ERR_ALIGN;
  AdamWState as{(uint16_t*)W, p->ld_w ? p->ld_w : p->d, exp_avg, exp_avg_sq, W_master};
  return backward_impl(p, nullptr, H, W, targets, lse, n_valid, grad_loss, dH, nullptr, nullptr, &as, &c,
                       workspace, workspace_bytes, stream);
}

lce_status_t lce_kd_workspace_size(const lce_kd_problem_t* p, size_t* fwd_bytes, size_t* bwd_bytes) {
  KdPlan k;
  lce_status_t st = make_kd_plan(p, &k);
  if (st != LCE_OK) return st;
  if (fwd_bytes) *fwd_bytes = k.fwd_bytes;
  if (bwd_bytes) *bwd_bytes = k.bwd_bytes;
  return LCE_OK;
}

lce_status_t lce_kd_forward(const lce_kd_problem_t* p, const void* Hs, const void* Ws, const void* Ht,
                            const void* Wt, const void* targets, float* loss, float* lse_s, float* lse_t,
                            int32_t* n_valid, int32_t* dev_status, void* workspace, size_t workspace_bytes,
                            void* stream) {
  return kd_forward_impl(p, Hs, Ws, Ht, Wt, targets, loss, lse_s, lse_t, n_valid, dev_status, workspace,
                         workspace_bytes, stream);
}

lce_status_t lce_kd_forward_backward(const lce_kd_problem_t* p, const void* Hs, const void* Ws, const void* Ht,
                                     const void* Wt, const void* targets, const float* grad_loss, float* loss,
                                     float* lse_s, float* lse_t, int32_t* n_valid, int32_t* dev_status, void* dHs,
                                     void* dWs, void* workspace, size_t workspace_bytes, void* stream) {
  return kd_fused_impl(p, Hs, Ws, Ht, Wt, targets, grad_loss, loss, lse_s, lse_t, n_valid, dev_status, dHs, dWs,
                       workspace, workspace_bytes, stream);
}

lce_status_t lce_kd_workspace_size_fused(const lce_kd_problem_t* p, size_t* bytes) {
  KdPlan k;
  lce_status_t st = make_kd_plan(p, &k);
  if (st != LCE_OK) return st;
  if (bytes) *bytes = k.fused_bytes;
  return LCE_OK;
}

lce_status_t lce_kd_backward(const lce_kd_problem_t* p, const void* Hs, const void* Ws, const void* Ht,
                             const void* Wt, const void* targets, const float* lse_s, const float* lse_t,
                             const int32_t* n_valid, const float* grad_loss, void* dHs, void* dWs,
                             void* workspace, size_t workspace_bytes, void* stream) {
  KdPlan k;
  lce_status_t st = make_kd_plan(p, &k);
  if (st != LCE_OK) return st;
  if (!dWs) return LCE_ERR_NULL;
  if (!aligned16(dWs)) return LCE_ERR_ALIGN;
  if (p->n > 0 && (!Ht || !Wt || !lse_t)) return LCE_ERR_NULL;
  if (p->n > 0 && (!aligned16(Ht) || !aligned16(Wt))) return LCE_ERR_ALIGN;
  const KdArgs kd{(const uint16_t*)Ht, k.t.ldh, (const uint16_t*)Wt, k.t.ldw, (int)k.t.d, lse_t, k.scale2, k.inv_t,
                  nullptr};
  return backward_impl(&k.ps, nullptr, Hs, Ws, targets, lse_s, n_valid, grad_loss, dHs, nullptr, (uint16_t*)dWs,
                       nullptr, nullptr, workspace, workspace_bytes, stream, &kd);
}

lce_status_t lce_timing_enable(int on) {
  std::lock_guard<std::mutex> lk(g_timing.mu);
  if (on) {
    if (g_timing.ev.empty()) {
      g_timing.ev.resize(2 * Timing::kPool);
      g_timing.kind.assign(Timing::kPool, 0);
      for (auto& e : g_timing.ev)
        if (hipEventCreate(&e) != hipSuccess) {
          g_timing.ev.clear();
          return LCE_ERR_HIP;
        }
    }
    g_timing.used = 0;
    g_timing.on = true;
  } else {
    g_timing.on = false;
  }
  return LCE_OK;
}

int lce_timing_kernel_count(void) { return K_COUNT; }

const char* lce_timing_kernel_name(int k) { return (k >= 0 && k < K_COUNT) ? kKernelNames[k] : nullptr; }

lce_status_t lce_timing_read(int k, double* total_ms, int64_t* launches) {
  if (k < 0 || k >= K_COUNT) return LCE_ERR_ARG;
  if (!total_ms || !launches) return LCE_ERR_NULL;
  std::lock_guard<std::mutex> lk(g_timing.mu);
  double tot = 0.0;
  int64_t cnt = 0;
  for (int i = 0; i < g_timing.used; ++i) {
    if (g_timing.kind[i] != k) continue;
    if (hipEventSynchronize(g_timing.ev[2 * i + 1]) != hipSuccess) return LCE_ERR_HIP;
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, g_timing.ev[2 * i], g_timing.ev[2 * i + 1]) != hipSuccess) return LCE_ERR_HIP;
    tot += ms;
    ++cnt;
  }
  *total_ms = tot;
  *launches = cnt;
  return LCE_OK;
}

}  // extern "C"
