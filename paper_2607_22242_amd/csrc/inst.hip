// inst.hip -- explicit instantiations of the kernels for the tool counts
// INST_LO..INST_HI (set on the compiler command line), so that the 40
// instantiations compile in parallel translation units.
#include "kernels.h"

#ifndef INST_LO
#error "INST_LO and INST_HI must be defined"
#endif

namespace devmap {

#define DEVMAP_INST(N)                                                            \
  template hipError_t launch_search_n<N>(const SearchArgs&, hipStream_t);         \
  template hipError_t launch_eval_n<N>(const uint32_t*, const uint64_t*, int64_t, \
                                       uint64_t, int64_t*, uint32_t, hipStream_t); \
  template hipError_t launch_bound_n<N>(const uint32_t*, uint32_t, uint64_t, int64_t, \
                                        uint32_t, uint32_t*, uint2*, hipStream_t);

#if INST_LO <= 1 && 1 <= INST_HI
DEVMAP_INST(1)
#endif
#if INST_LO <= 2 && 2 <= INST_HI
DEVMAP_INST(2)
#endif
#if INST_LO <= 3 && 3 <= INST_HI
DEVMAP_INST(3)
#endif
#if INST_LO <= 4 && 4 <= INST_HI
DEVMAP_INST(4)
#endif
#if INST_LO <= 5 && 5 <= INST_HI
DEVMAP_INST(5)
#endif
#if INST_LO <= 6 && 6 <= INST_HI
DEVMAP_INST(6)
#endif
#if INST_LO <= 7 && 7 <= INST_HI
DEVMAP_INST(7)
#endif
#if INST_LO <= 8 && 8 <= INST_HI
DEVMAP_INST(8)
#endif
#if INST_LO <= 9 && 9 <= INST_HI
DEVMAP_INST(9)
#endif
#if INST_LO <= 10 && 10 <= INST_HI
DEVMAP_INST(10)
#endif
#if INST_LO <= 11 && 11 <= INST_HI
DEVMAP_INST(11)
#endif
#if INST_LO <= 12 && 12 <= INST_HI
DEVMAP_INST(12)
#endif
#if INST_LO <= 13 && 13 <= INST_HI
DEVMAP_INST(13)
#endif
#if INST_LO <= 14 && 14 <= INST_HI
DEVMAP_INST(14)
#endif
#if INST_LO <= 15 && 15 <= INST_HI
DEVMAP_INST(15)
#endif
#if INST_LO <= 16 && 16 <= INST_HI
DEVMAP_INST(16)
#endif
#if INST_LO <= 17 && 17 <= INST_HI
DEVMAP_INST(17)
#endif
#if INST_LO <= 18 && 18 <= INST_HI
DEVMAP_INST(18)
#endif
#if INST_LO <= 19 && 19 <= INST_HI
DEVMAP_INST(19)
#endif
#if INST_LO <= 20 && 20 <= INST_HI
DEVMAP_INST(20)
#endif
#if INST_LO <= 21 && 21 <= INST_HI
DEVMAP_INST(21)
#endif
#if INST_LO <= 22 && 22 <= INST_HI
DEVMAP_INST(22)
#endif
#if INST_LO <= 23 && 23 <= INST_HI
DEVMAP_INST(23)
#endif
#if INST_LO <= 24 && 24 <= INST_HI
DEVMAP_INST(24)
#endif
#if INST_LO <= 25 && 25 <= INST_HI
DEVMAP_INST(25)
#endif
#if INST_LO <= 26 && 26 <= INST_HI
DEVMAP_INST(26)
#endif
#if INST_LO <= 27 && 27 <= INST_HI
DEVMAP_INST(27)
#endif
#if INST_LO <= 28 && 28 <= INST_HI
DEVMAP_INST(28)
#endif
#if INST_LO <= 29 && 29 <= INST_HI
DEVMAP_INST(29)
#endif
#if INST_LO <= 30 && 30 <= INST_HI
DEVMAP_INST(30)
#endif
#if INST_LO <= 31 && 31 <= INST_HI
DEVMAP_INST(31)
#endif
#if INST_LO <= 32 && 32 <= INST_HI
DEVMAP_INST(32)
#endif
#if INST_LO <= 33 && 33 <= INST_HI
DEVMAP_INST(33)
#endif
#if INST_LO <= 34 && 34 <= INST_HI
DEVMAP_INST(34)
#endif
#if INST_LO <= 35 && 35 <= INST_HI
DEVMAP_INST(35)
#endif
#if INST_LO <= 36 && 36 <= INST_HI
DEVMAP_INST(36)
#endif
#if INST_LO <= 37 && 37 <= INST_HI
DEVMAP_INST(37)
#endif
#if INST_LO <= 38 && 38 <= INST_HI
DEVMAP_INST(38)
#endif
#if INST_LO <= 39 && 39 <= INST_HI
DEVMAP_INST(39)
#endif
#if INST_LO <= 40 && 40 <= INST_HI
DEVMAP_INST(40)
#endif

}  // namespace devmap
