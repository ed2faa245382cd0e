"""MI355X-native beam-search decode step (FastSeq, arXiv 2106.04718)."""
