"""MI355X-native batched query-time search of NeuRoute (arXiv 2608.15438)."""
