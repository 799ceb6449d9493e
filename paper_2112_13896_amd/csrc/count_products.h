// Product counter of the counting build (compiled with -DCS_COUNT_PRODUCTS
// into libcs_count.so).  Every multiply-route-sum kernel adds the number of
// weight x activation products it forms for live list entries; the total is
// then the number of pairs with a non-zero activation and a non-zero packed
// weight, which for a packing without holes is the count of non-zero
// (weight, activation) pairs of the dense layer (Section 3.2, Figure 1: the
// work is proportional to the product of the two densities).  A kernel that
// multiplied dense rows, or entries past a list's count, would count more.
// In the product build the macro expands to nothing.
#pragma once

#ifdef CS_COUNT_PRODUCTS
__device__ unsigned long long cs_products_formed;
#define CS_COUNT_PRODUCTS_ADD(n)                                                         \
  do {                                                                                  \
    const int cs_n_ = (n);                                                              \
    if (cs_n_ > 0) atomicAdd(&cs_products_formed, (unsigned long long)cs_n_);           \
  } while (0)
#else
#define CS_COUNT_PRODUCTS_ADD(n) \
  do {                           \
  } while (0)
#endif
