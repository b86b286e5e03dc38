"""MI355X-native datapath executor of Purlin (arXiv 2609.36954)."""
