// Which build of the kernels a translation unit compiles.
//
// The draw kernels address theta and phi with 32-bit row handles.  With
// LDA_WIDE_TABLES 0 (the default) a handle is the row's byte offset and a
// table is read through a buffer resource, so tables stay below 4 GiB.  With
// LDA_WIDE_TABLES 1 a handle is the row index and every load forms a 64-bit
// address, so tables may be of any size; that build lives in its own
// translation unit and namespace (LDA_NS), next to the default one.
#pragma once

#ifndef LDA_WIDE_TABLES
#define LDA_WIDE_TABLES 0
#endif

#if LDA_WIDE_TABLES
#define LDA_NS lda_wide
#else
#define LDA_NS lda
#endif
