"""MI355X-native Turbo-Muon orthogonalization (AOL pre-conditioning + quintic Newton-Schulz)."""
