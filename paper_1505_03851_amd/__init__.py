"""MI355X-native per-token LDA topic draw with butterfly-patterned partial
sums (Steele and Tristan, arXiv 1505.03851)."""
