// Device-side building blocks shared by the BLA kernels (gfx950 / CDNA4).
//
// Matrix-core convention used everywhere.  Every contraction is computed with
// 16x16 output tiles on the matrix cores: bf16 operands use
// v_mfma_f32_16x16x32_bf16, float32 operands use eight v_mfma_f32_16x16x4_f32.
// For a 64-lane wave, lane l has group g = l / 16 and index r = l % 16.
//
//  * Accumulator tile (floatx4): lane (g, r) holds rows 4g+0..3 of column r.
//  * Operand fragment for reduction block kb (32 reduction indices): lane (g, r)
//    holds 8 values for row r (A operand) or column r (B operand), element e at
//    reduction index  k(e) = 32 kb + 16 (e / 4) + 4 g + (e % 4).
//    The same k(e) is used for A and B, so the products pair up correctly
//    whatever order the hardware walks the reduction in.
//  * With this k(e), two stacked accumulator tiles (rows 32kb..32kb+15 and
//    32kb+16..32kb+31) ARE the B fragment of the next contraction over those
//    rows (and, for a transposed state, the A fragment), so chains of
//    contractions pass their intermediates in registers without a shuffle.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace bla {

typedef __bf16 bf16;
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef float floatx8 __attribute__((ext_vector_type(8)));
typedef int intx4 __attribute__((ext_vector_type(4)));
typedef _Float16 halfx4 __attribute__((ext_vector_type(4)));

template <typename T> struct Frag;
template <> struct Frag<bf16> { typedef bf16x8 type; typedef bf16x4 half; };
template <> struct Frag<float> { typedef floatx8 type; typedef floatx4 half; };

__device__ __forceinline__ floatx4 mma(bf16x8 a, bf16x8 b, floatx4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ floatx4 mma(floatx8 a, floatx8 b, floatx4 c)
{
#pragma unroll
    for (int e = 0; e < 8; ++e) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[e], b[e], c, 0, 0, 0);
    return c;
}

__device__ __forceinline__ floatx4 zero4() { return floatx4{0.f, 0.f, 0.f, 0.f}; }

// A uniform pointer the optimiser cannot see through (no code is emitted).  Re-deriving a
// table pointer this way once per loop iteration keeps the table's fragments from being
// hoisted out of the loop into registers (which spills when the tables are large).  The
// pointer itself is not passed through the asm statement, only a zero offset added to it:
// the compiler still sees that it addresses global memory (a kernel argument) and emits
// global loads, not flat ones (a flat load counts against the LDS wait counter as well, so
// every wait for an LDS read would also wait for the table loads in flight).
template <typename P> __device__ __forceinline__ const P* opaque(const P* p)
{
    int zero = 0;
    asm volatile("" : "+s"(zero));
    return p + zero;
}

// A lane value the optimiser cannot see through (no code is emitted).  Lane indices
// re-derived this way at the top of each iteration of a chunk loop make the per-lane
// addresses computed from them loop-variant, so they are recomputed inside the loop (a few
// vector instructions) instead of being hoisted out and kept live across it, which spilled
// them to scratch; every reload from scratch then waited for all outstanding memory loads.
__device__ __forceinline__ int opaque_lane(int x)
{
    asm volatile("" : "+v"(x));
    return x;
}

// Stores and loads through a generic pointer that is known to address LDS (or global
// memory): the explicit address space gives ds_write / global_load instructions instead of
// flat ones (a flat access counts against both the LDS and the memory wait counters, so
// each wait for one waits for the other as well).
template <typename V, typename P> __device__ __forceinline__ void st_lds(P* p, V x)
{
    *(__attribute__((address_space(3))) V*)p = x;
}
template <typename V, typename P> __device__ __forceinline__ V ld_global(const P* p)
{
    return *(const __attribute__((address_space(1))) V*)p;
}

template <typename T> __device__ __forceinline__ typename Frag<T>::type zero_frag()
{
    typename Frag<T>::type f;
#pragma unroll
    for (int e = 0; e < 8; ++e) f[e] = (T)0.f;
    return f;
}

template <typename T> __device__ __forceinline__ typename Frag<T>::half zero_half()
{
    typename Frag<T>::half f;
#pragma unroll
    for (int e = 0; e < 4; ++e) f[e] = (T)0.f;
    return f;
}

__device__ __forceinline__ bf16x8 join(bf16x4 a, bf16x4 b)
{
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}
__device__ __forceinline__ floatx8 join(floatx4 a, floatx4 b)
{
    return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}

typedef short shortx4 __attribute__((ext_vector_type(4)));

// Transposing LDS read: within each 16-lane group, lane 4a+b supplies the address
// of 4 consecutive elements; lane 4b'+c receives element c of lane 4a+b' for a = 0..3.
__device__ __forceinline__ bf16x4 ld_tr(const bf16* p)
{
    shortx4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) shortx4*)p);
    return __builtin_bit_cast(bf16x4, v);
}

// Operand fragment for rows x0..x0+15 (lane r) and reduction block kb from an LDS
// tile stored reduction-major, M[k][x] with row length ld: the fragment's element e
// of lane (g, r) is M[k(e)][x0 + r], k(e) = 32kb + 16(e/4) + 4g + e%4.
__device__ __forceinline__ bf16x8 ld_frag_tr(const bf16* M, int ld, int x0, int kb, int g, int r)
{
    const bf16* p = M + (size_t)(32 * kb + 4 * g + (r >> 2)) * ld + x0 + 4 * (r & 3);
    return join(ld_tr(p), ld_tr(p + (size_t)16 * ld));
}

// Fragment-ordered rows.  An operand fragment takes the reduction indices 32kb + 4g .. + 3
// and 32kb + 16 + 4g .. + 3 of a row (the order two stacked accumulator tiles give).  A table
// whose rows are stored with the 4-column group 16h + 4j (h = 0, 1; j = 0..3) of every block
// of 32 columns moved to 8j + 4h holds those eight indices next to each other, so the
// fragment is one 16-byte LDS read instead of two 8-byte reads 32 bytes apart (which gfx950
// serves at a quarter of the 16-byte rate).  frag_col maps a logical column (a multiple of 4)
// to its stored position.
__host__ __device__ constexpr int frag_col(int c)
{
    return (c & ~31) | (((c >> 2) & 3) << 3) | (((c >> 4) & 1) << 2);
}

// Fragment from a fragment-ordered row, or from a natural row with the reduction order
// k(e) = 32kb + 8g + e (both operands of a contraction must use the same order): one
// 16-byte read at 32kb + 8g.
__device__ __forceinline__ bf16x8 ld_frag16(const bf16* row, int kb, int g)
{
    return *reinterpret_cast<const bf16x8*>(row + 32 * kb + 8 * g);
}

// ld_frag16's fragment (reduction order 32kb + 8g + e) from an LDS row that is only 8-byte
// aligned: two 8-byte reads (the second volatile, as in ld_frag_2x8).
__device__ __forceinline__ bf16x8 ld_frag16_2x8(const bf16* row, int kb, int g)
{
    typedef const __attribute__((address_space(3))) bf16x4 lds4;
    lds4* a = (lds4*)(row + 32 * kb + 8 * g);
    return join(*a, *(const volatile __attribute__((address_space(3))) bf16x4*)(a + 1));
}

// Fragment of a natural row for the accumulator order (32kb + 4g .. + 3, 32kb + 16 + 4g ..
// + 3) as two separate 8-byte LDS reads.  The second read is volatile so that the two are not
// merged into one ds_read2_b64, which gfx950 serves at a quarter to half of the rate of two
// ds_read_b64 at these addresses.
__device__ __forceinline__ bf16x8 ld_frag_2x8(const bf16* row, int kb, int g)
{
    typedef const __attribute__((address_space(3))) bf16x4 lds4;
    lds4* a = (lds4*)(row + 32 * kb + 4 * g);
    return join(*a, *(const volatile __attribute__((address_space(3))) bf16x4*)(a + 4));
}

// Row-swizzled tables.  A table read both as row fragments (ld_frag_2x8: 16 rows, 8 bytes per
// lane) and transposed (ld_frag_tr: 8 consecutive rows per half wave) at a row stride of
// 8 (mod 64) dwords has no bank conflicts in its transposed reads, but its row-fragment reads
// put rows r and r + 8 on the same banks.  Storing the 4-element column groups of every row
// with bit 3 set at column XOR 8 moves those rows onto the other half of the banks; the eight
// rows of a transposed half wave share bit 3, so their reads stay conflict-free.
__host__ __device__ constexpr int swz_col(int row, int col) { return col ^ (((row >> 3) & 1) << 3); }

// ld_frag_2x8 on a swizzled table; row points at table row 16i + r.  The swizzle touches
// bit 3 of the column only, so it applies to the lane's part 4g and the block offsets 32kb
// and 16 stay immediate.
__device__ __forceinline__ bf16x8 ld_frag_2x8_sw(const bf16* row, int kb, int g, int r)
{
    typedef const __attribute__((address_space(3))) bf16x4 lds4;
    lds4* a = (lds4*)(row + ((4 * g) ^ ((r >> 3) << 3)) + 32 * kb);
    return join(*a, *(const volatile __attribute__((address_space(3))) bf16x4*)(a + 4));
}

// Row swizzle keyed on bit 2 of the row, for a table written as 16 x 16 accumulator tiles
// (8-byte pieces, one row per lane of a 16-lane group) and read as 16-byte row fragments.  An
// 8-byte LDS write serves 16 lanes per cycle over 32 banks, so at a row stride of 8 (mod 32)
// dwords the 16 rows of a tile fall on 4 bank groups (4-way conflicts); flipping bit 3 of the
// column in rows 4-7 and 12-15 of every 16 halves that, and unlike the bit-3 swizzle it keeps
// the 16-byte row-fragment reads of such a table conflict-free (both measured with the LDS
// bank-conflict counter on gfx950).
__host__ __device__ constexpr int swz4_col(int row, int col) { return col ^ (((row >> 2) & 1) << 3); }

// ld_frag16 on a swz4_col table; row points at table row 16i + r.  The lane's 8-element block
// 8g moves to 8(g ^ 1) in the rows the swizzle flips and stays one 16-byte read.
__device__ __forceinline__ bf16x8 ld_frag16_sw4(const bf16* row, int kb, int g, int r)
{
    return *reinterpret_cast<const bf16x8*>(row + 32 * kb + ((8 * g) ^ (((r >> 2) & 1) << 3)));
}

// ld_frag_tr on a swizzled table (rows 32kb + 4g + r/4 and 16 below: bit 3 is bit 1 of g;
// x0 is a multiple of 16).
__device__ __forceinline__ bf16x8 ld_frag_tr_sw(const bf16* M, int ld, int x0, int kb, int g, int r)
{
    const bf16* p = M + (size_t)(32 * kb + 4 * g + (r >> 2)) * ld + x0 + ((4 * (r & 3)) ^ ((g >> 1) << 3));
    return join(ld_tr(p), ld_tr(p + (size_t)16 * ld));
}

// Piece swizzle for tiles written as 16 x 16 accumulator tiles with 8-byte stores (one row per
// lane of a 16-lane group, 16 lanes per store cycle over 32 banks) and read only transposed
// (ld_tr: 8 rows of 32 bytes per half wave).  At a row stride of 8 x odd (mod 64) dwords the
// transposed reads are conflict-free, but the 16 rows of a store fall on 4 bank groups;
// XOR-ing the 4-element piece index inside each 16-column group with bits 2-3 of the row
// spreads them over all 32 banks, while each row keeps its 4 pieces in the same 32 bytes.
__host__ __device__ constexpr int pswz_col(int row, int col) { return col ^ (((row >> 2) & 3) << 2); }

// ld_frag_tr on a pswz_col table (x0 a multiple of 16): the rows 32kb + 4g + r/4 and 16 below
// have bits 2-3 equal to g.
__device__ __forceinline__ bf16x8 ld_frag_tr_ps(const bf16* M, int ld, int x0, int kb, int g, int r)
{
    const bf16* p = M + (size_t)(32 * kb + 4 * g + (r >> 2)) * ld + x0 + 4 * ((r & 3) ^ g);
    return join(ld_tr(p), ld_tr(p + (size_t)16 * ld));
}

// ld_frag_tr on a tile whose columns are fragment-ordered (4-column groups stay contiguous,
// so each lane's 4 consecutive elements are still one 8-byte read).
__device__ __forceinline__ bf16x8 ld_frag_tr_fo(const bf16* M, int ld, int x0, int kb, int g, int r)
{
    const bf16* p = M + (size_t)(32 * kb + 4 * g + (r >> 2)) * ld + frag_col(x0 + 4 * (r & 3));
    return join(ld_tr(p), ld_tr(p + (size_t)16 * ld));
}

// Four consecutive elements as a vector (pointer 4-element aligned).
template <typename T> __device__ __forceinline__ typename Frag<T>::half ld4(const T* p)
{
    return *reinterpret_cast<const typename Frag<T>::half*>(p);
}

// Fragment of a row-major matrix whose reduction index is contiguous in memory:
// `row` points at the lane's row (A) or column (B); k0 = 32 kb.
template <typename T>
__device__ __forceinline__ typename Frag<T>::type ld_frag(const T* row, int k0, int g)
{
    return join(ld4<T>(row + k0 + 4 * g), ld4<T>(row + k0 + 16 + 4 * g));
}

// Same, with the upper half (reduction indices k0+16..k0+31) replaced by zeros.
template <typename T>
__device__ __forceinline__ typename Frag<T>::type ld_frag_lo(const T* row, int k0, int g)
{
    return join(ld4<T>(row + k0 + 4 * g), zero_half<T>());
}

__device__ __forceinline__ bf16x4 cvt4(floatx4 x, bf16)
{
    bf16x4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = (bf16)x[e];
    return r;
}
__device__ __forceinline__ floatx4 cvt4(floatx4 x, float) { return x; }

// Two stacked accumulator tiles -> operand fragment (see the header comment).
template <typename T>
__device__ __forceinline__ typename Frag<T>::type frag_from_acc(floatx4 lo, floatx4 hi)
{
    return join(cvt4(lo, T()), cvt4(hi, T()));
}

// Store four floats as four consecutive elements of type T.
template <typename T> __device__ __forceinline__ void st4(T* p, floatx4 x)
{
    *reinterpret_cast<typename Frag<T>::half*>(p) = cvt4(x, T());
}

// Same, from LDS through an LDS-typed pointer: a load that cannot be merged with a global
// load of another branch into one generic (flat) load.
template <typename T> __device__ __forceinline__ typename Frag<T>::half ld4_lds(const T* p)
{
    typedef typename Frag<T>::half H;
    return *(const __attribute__((address_space(3))) H*)p;
}

__device__ __forceinline__ floatx4 ld4f(const float* p) { return *reinterpret_cast<const floatx4*>(p); }
__device__ __forceinline__ void st4f(float* p, floatx4 x) { *reinterpret_cast<floatx4*>(p) = x; }

// Up-convert a 4-vector of T to float.
__device__ __forceinline__ floatx4 to_f4(bf16x4 x)
{
    floatx4 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) r[e] = (float)x[e];
    return r;
}
__device__ __forceinline__ floatx4 to_f4(floatx4 x) { return x; }

// Reductions over the four 16-lane rows of a wave: lane (g, r) receives the result for
// column r over g = 0..3.  The two lane-swap instructions exchange rows 0,1 <-> 2,3 and
// 0 <-> 1, 2 <-> 3 in registers; each pair (kept, received) is the pair (x[l], x[l^32]) or
// (x[l], x[l^16]) in some order, so every lane of a column ends with identical bits.
__device__ __forceinline__ float rows_max(float x)
{
    const unsigned u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    const float y = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
    const unsigned v = __float_as_uint(y);
    const auto b = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows_sum(float x)
{
    const unsigned u = __float_as_uint(x);
    const auto a = __builtin_amdgcn_permlane32_swap(u, u, false, false);
    const float y = __uint_as_float(a[0]) + __uint_as_float(a[1]);
    const unsigned v = __float_as_uint(y);
    const auto b = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Complex twiddle of four accumulator rows with a half-precision phase (c, n):
//     (re, im) <- (c re + n im, c im - n re)        (NEG: n replaced by -n)
// Each product takes its half-precision factor as a mixed-precision FMA operand, so the
// phase needs no conversion (the product with the zero addend stays an FMA).
template <bool NEG>
__device__ __forceinline__ void twiddle_h(halfx4 c, halfx4 n, floatx4& re, floatx4& im)
{
    floatx4 r, i;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        const float cf = (float)c[e], nf = NEG ? -(float)n[e] : (float)n[e];
        r[e] = __builtin_fmaf(cf, re[e], __builtin_fmaf(nf, im[e], 0.f));
        i[e] = __builtin_fmaf(cf, im[e], __builtin_fmaf(-nf, re[e], 0.f));
    }
    re = r;
    im = i;
}

// cos and sin of the absolute phase m w P (w = 2 pi / T) for the anchored slots of
// Sec. 3.3, from the reciprocal period rT = 1 / T.  m P is an exact integer in double;
// the revolutions m P / T are reduced to [0, 1) in double before the single-precision
// sincos, so a position far past the period keeps the phase accuracy of a small one.
__device__ __forceinline__ void anchor_phase(int m, long long P, double rT, float& c, float& s)
{
    const double x = (double)m * (double)P * rT;
    const float f = (float)(x - floor(x));
    sincospif(2.f * f, &s, &c);
}

}  // namespace bla
