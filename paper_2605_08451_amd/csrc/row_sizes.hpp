// row_sizes.hpp -- row DFT sizes with a register-resident kernel.
//
// X(m, M1, M2): m = M1 * M2 with M1 >= M2, both small radices, as balanced as
// possible.  The plan rounds a document's row size up to the next entry of this
// list while the list covers it (every entry is a 2^a 3^b 5^c number); longer
// rows use the generic row kernel.
#pragma once

#define RUBICONV_ROW_SIZES(X)                                                                  \
    X(1, 1, 1) X(2, 2, 1) X(3, 3, 1) X(4, 2, 2) X(5, 5, 1) X(6, 3, 2) X(8, 4, 2) X(9, 3, 3)    \
    X(10, 5, 2) X(12, 4, 3) X(15, 5, 3) X(16, 4, 4) X(18, 6, 3) X(20, 5, 4) X(24, 6, 4)        \
    X(25, 5, 5) X(27, 9, 3) X(30, 6, 5) X(32, 8, 4) X(36, 6, 6) X(40, 8, 5) X(45, 9, 5)        \
    X(48, 8, 6) X(50, 10, 5) X(54, 9, 6) X(60, 10, 6) X(64, 8, 8) X(72, 9, 8) X(75, 15, 5)     \
    X(80, 10, 8) X(81, 9, 9) X(90, 10, 9) X(96, 12, 8) X(100, 10, 10) X(108, 12, 9)            \
    X(120, 12, 10) X(128, 16, 8) X(135, 15, 9) X(144, 12, 12) X(150, 15, 10) X(160, 16, 10)    \
    X(180, 15, 12) X(192, 16, 12) X(225, 15, 15) X(240, 16, 15) X(256, 16, 16)

namespace rubiconv {

constexpr int kMaxFastM = 256;

// Smallest listed size >= v, or 0 if v exceeds the list.
inline int fast_row_size(int v) {
#define RUBICONV_PICK(m, a, b) \
    if (v <= (m)) return (m);
    RUBICONV_ROW_SIZES(RUBICONV_PICK)
#undef RUBICONV_PICK
    return 0;
}

}  // namespace rubiconv
