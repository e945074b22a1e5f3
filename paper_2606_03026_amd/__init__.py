"""MI355X-native spike-gated INT8 projection (placeholder until the binding lands)."""
