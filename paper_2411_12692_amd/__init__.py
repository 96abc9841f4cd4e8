"""MI355X-native SparseInfer decode path (placeholder until the binding lands)."""
