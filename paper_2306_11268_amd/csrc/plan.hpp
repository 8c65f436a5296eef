// Two-level decomposition of a length-N DFT, N = N1 * N2, used by the tile kernels.
//
// A vector of length N is held as an N1 x N2 array in shared memory, element
// (x, j) in slot x*N2 + j.  Its transform is carried out in two register steps:
//
//   A-step: N2 "A-items" (one per j); item j holds the N1 elements (x, j),
//           x < N1 (slots j + N2*x), and runs a length-N1 DFT over x.
//   B-step: N1 "B-items" (one per k1); item k1 holds the N2 elements
//           (k1, j), j < N2 (slots N2*k1 + j), optionally multiplies by the
//           Cooley-Tukey twiddles exp(-2*pi*i*k1*j/N), and runs a length-N2
//           DFT over j.  Element k2 of item k1 is frequency freq(k1, k2).
//
// Every item reads and writes its own slots, so both steps work in place
// and items can be processed one at a time; slot addresses are affine in the
// element index.  The inverse transform runs the steps in the opposite order
// with conjugated roots.  The natural (spatial) position of element (x, j):
//
// CT  (Cooley-Tukey):   pos(x, j) = j + N2*x (the slot itself),  freq = k1 + N1*k2
// PFA (Good-Thomas, gcd(N1,N2) = 1, no twiddles):
//                       pos(x, j) = (N2*x + N1*j) mod N,        freq = CRT(k1 mod N1, k2 mod N2)
//
// Slot order as a storage order: a field whose rows and columns are both
// stored in slot order (stored index s along an axis holds natural position
// pos_of_slot(s)) has the elements of A-item j at the stored indices
// j + N2*x, a constant stride, for either plan; in natural order the
// Good-Thomas positions wrap around N once per item.
#pragma once

#include "codelets.hpp"

namespace lr {

template <int N>
struct Roots {
  static constexpr RootTable<N> table = make_root_table<N>();
};

template <int N1_, int N2_, bool PFA_>
struct Plan2 {
  static constexpr int N1 = N1_;
  static constexpr int N2 = N2_;
  static constexpr int N = N1_ * N2_;
  static constexpr bool PFA = PFA_;
  static constexpr int E1 = PFA_ ? N2_ * inv_mod(N2_ % N1_, N1_) : 0;
  static constexpr int E2 = PFA_ ? N1_ * inv_mod(N1_ % N2_, N2_) : 0;
  static constexpr int U1 = PFA_ ? inv_mod(N2_ % N1_, N1_) : 0;
  static constexpr int U2 = PFA_ ? inv_mod(N1_ % N2_, N2_) : 0;
  static_assert(!PFA_ || (inv_mod(N2_ % N1_, N1_) > 0 && inv_mod(N1_ % N2_, N2_) > 0),
                "PFA needs coprime factors");

  // Slot of element x of A-item j, and of element j of B-item k1.
  LR_HD static int a_slot(int j, int x) { return j + N2 * x; }
  LR_HD static int b_slot(int k1, int j) { return N2 * k1 + j; }

  // Natural position of element (x, j), written as pos_base(j) + N2*x (mod N).
  LR_HD static int pos_base(int j) { return PFA ? (N1 * j) % N : j; }
  LR_HD static int pos_at(int base, int x) {
    if (PFA) {
      const int p = base + N2 * x;
      return p >= N ? p - N : p;
    }
    return base + N2 * x;
  }
  LR_HD static int pos(int x, int j) { return pos_at(pos_base(j), x); }
  // Natural position held by slot s (inverse of slot_of_pos).
  LR_HD static int pos_of_slot(int s) { return pos(s / N2, s % N2); }
  // Slot holding natural position p.
  LR_HD static int slot_of_pos(int p) {
    if (PFA) return ((p % N1) * U1 % N1) * N2 + (p % N2) * U2 % N2;
    return p;
  }
  // Slot of natural position p advanced one position at a time, without
  // divisions: under the Good-Thomas map the slot is (s1, s2) =
  // ((p mod N1) * U1 mod N1, (p mod N2) * U2 mod N2), and p + 1 adds (U1, U2).
  struct Walk {
    int s1;
    int s2;
  };
  LR_HD static Walk walk(int p) { return PFA ? Walk{(p % N1) * U1 % N1, (p % N2) * U2 % N2} : Walk{p, 0}; }
  LR_HD static int walk_slot(const Walk& w) { return PFA ? w.s1 * N2 + w.s2 : w.s1; }
  LR_HD static void walk_next(Walk& w) {
    if (PFA) {
      w.s1 += U1;
      if (w.s1 >= N1) w.s1 -= N1;
      w.s2 += U2;
      if (w.s2 >= N2) w.s2 -= N2;
    } else {
      ++w.s1;
    }
  }
  // Frequency index of element k2 of B-item k1 and its inverse (slot of frequency f).
  LR_HD static int freq(int k1, int k2) {
    return PFA ? (k1 * E1 + k2 * E2) % N : k1 + N1 * k2;
  }
  LR_HD static int slot_of_freq(int f) { return b_slot(f % N1, PFA ? f % N2 : f / N1); }

  // Forward-direction twiddle of B-item k1, element j: exp(-2*pi*i*k1*j/N).
  LR_HD static float2 twiddle(int k1, int j) { return Roots<N>::table.w[k1 * j]; }
};

// Plans by FFT length.  N1 is the length of the A-step transforms (one A-item
// per thread), N2 that of the B-step ones.  Sizes without an entry are
// rejected by the host code.  The Good-Thomas map is used where the factors
// are coprime (no twiddles).  Row and column passes may use different plans
// (RowPlanFor); the transfer-function tables are built for each.
template <int N> struct PlanFor;
template <> struct PlanFor<64>   { using type = Plan2<8, 8, false>; };
template <> struct PlanFor<100>  { using type = Plan2<25, 4, true>; };
template <> struct PlanFor<128>  { using type = Plan2<16, 8, false>; };
template <> struct PlanFor<200>  { using type = Plan2<25, 8, true>; };
template <> struct PlanFor<256>  { using type = Plan2<16, 16, false>; };
template <> struct PlanFor<350>  { using type = Plan2<25, 14, true>; };
template <> struct PlanFor<400>  { using type = Plan2<25, 16, true>; };
template <> struct PlanFor<500>  { using type = Plan2<25, 20, false>; };
template <> struct PlanFor<512>  { using type = Plan2<32, 16, false>; };
template <> struct PlanFor<1000> { using type = Plan2<25, 40, false>; };
template <> struct PlanFor<1024> { using type = Plan2<32, 32, false>; };

template <int N>
struct RowPlanFor {
  using type = typename PlanFor<N>::type;
};

}  // namespace lr
